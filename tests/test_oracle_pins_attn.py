"""Pins of the oracle's INT8 key/value cache and one-token attention (Sec. 4,
further speed-ups: INT8 key/value cache; Sec. 2: four query heads share one
key/value head of 256; eq. attnffn55 / attnffn1010 for the attention layer
sets).

The attention is pinned to torch's own scaled-dot-product attention in
binary64 (a library routine that shares nothing with the oracle's C loops) and
to closed forms: one cached row returns its value, equal keys average the
values, a shift of every key by one vector changes nothing, two keys give the
logistic weight.  A transposed key, a dropped 1/sqrt(d) scale, a missing
normalisation or a wrong window start each fail one of them.
"""

import math

import numpy as np
import pytest
import torch

import oracle
from paper_2608_28003_amd import synth

DH = oracle.HEAD_DIM
H = oracle.N_Q_HEADS


def rng(seed):
    return np.random.default_rng(seed)


def sdpa(q, k, v, scale):
    """torch's attention for one query token: q (h, dh), k / v (t, dh), the
    one key/value head shared by every query head."""
    qt = torch.from_numpy(q)[None, :, None, :]            # 1, h, 1, dh
    h = q.shape[0]
    kt = torch.from_numpy(k)[None, None].expand(1, h, -1, -1)
    vt = torch.from_numpy(v)[None, None].expand(1, h, -1, -1)
    out = torch.nn.functional.scaled_dot_product_attention(qt, kt, vt, scale=scale)
    return out[0, :, 0, :].numpy()


@pytest.mark.parametrize("t", [1, 2, 17, 300])
def test_attn_decode_matches_torch_sdpa(t):
    r = rng(10 + t)
    q = r.standard_normal((H, DH))
    k = r.standard_normal((t, DH))
    v = r.standard_normal((t, DH))
    out = oracle.attn_decode(q, k, v)
    ref = sdpa(q, k, v, oracle.ATTN_SCALE)
    np.testing.assert_allclose(out, ref, rtol=1e-12, atol=1e-12)
    # power: without the 1/sqrt(d) scale, or with transposed key rows, the
    # answer moves far outside that tolerance
    if t > 1:
        assert np.abs(oracle.attn_decode(q, k, v, scale=1.0) - ref).max() > 1e-3
        kt = np.ascontiguousarray(k.reshape(-1)[np.arange(t * DH).reshape(DH, t).T.reshape(-1)].reshape(t, DH))
        assert np.abs(oracle.attn_decode(q, kt, v) - ref).max() > 1e-3


def test_single_row_returns_its_value():
    r = rng(1)
    q = r.standard_normal((H, DH)) * 5
    k = r.standard_normal((1, DH))
    v = r.standard_normal((1, DH))
    out = oracle.attn_decode(q, k, v)
    np.testing.assert_array_equal(out, np.repeat(v, H, axis=0))


def test_equal_keys_average_the_values():
    r = rng(2)
    q = r.standard_normal((H, DH))
    k = np.repeat(r.standard_normal((1, DH)), 37, axis=0)
    v = r.standard_normal((37, DH))
    out = oracle.attn_decode(q, k, v)
    np.testing.assert_allclose(out, np.repeat(v.mean(0, keepdims=True), H, axis=0), rtol=0, atol=1e-14)


def test_two_keys_give_the_logistic_weight():
    r = rng(3)
    q = r.standard_normal((1, DH))
    k = r.standard_normal((2, DH))
    v = r.standard_normal((2, DH))
    s = [float(q[0] @ k[i]) / 16.0 for i in range(2)]
    p0 = 1.0 / (1.0 + math.exp(s[1] - s[0]))
    np.testing.assert_allclose(oracle.attn_decode(q, k, v)[0], p0 * v[0] + (1 - p0) * v[1],
                               rtol=1e-13, atol=1e-13)


def test_shift_of_every_key_changes_nothing():
    """q.(k_t + c) adds the same q.c to every score of a head."""
    r = rng(4)
    q = r.standard_normal((H, DH))
    k = r.standard_normal((50, DH))
    v = r.standard_normal((50, DH))
    c = r.standard_normal(DH) * 3
    np.testing.assert_allclose(oracle.attn_decode(q, k + c, v), oracle.attn_decode(q, k, v),
                               rtol=1e-11, atol=1e-12)


def test_row_order_and_head_independence():
    r = rng(5)
    q = r.standard_normal((H, DH))
    k = r.standard_normal((40, DH))
    v = r.standard_normal((40, DH))
    out = oracle.attn_decode(q, k, v)
    perm = r.permutation(40)
    np.testing.assert_allclose(oracle.attn_decode(q, k[perm], v[perm]), out, rtol=1e-12, atol=1e-13)
    for i in range(H):
        np.testing.assert_array_equal(oracle.attn_decode(q[i:i + 1], k, v)[0], out[i])


def test_large_scores_stay_finite():
    r = rng(6)
    q = r.standard_normal((H, DH)) * 300
    k = r.standard_normal((20, DH)) * 300
    v = r.standard_normal((20, DH))
    out = oracle.attn_decode(q, k, v)
    assert np.isfinite(out).all()
    np.testing.assert_allclose(out, sdpa(q, k, v, oracle.ATTN_SCALE), rtol=1e-9, atol=1e-9)


def test_kv_quantize_is_the_per_token_rule_without_smoothing():
    r = rng(7)
    x = synth.to_bf16_bits((r.standard_normal((64, DH)) * np.exp(r.standard_normal((64, 1)))).astype(np.float32))
    x[5] = 0
    q, s = oracle.kv_quantize(x)
    q2, s2 = oracle.quantize_act(x, None)
    np.testing.assert_array_equal(q, q2)
    np.testing.assert_array_equal(s, s2)
    xf = oracle.bf16_to_f32(x).astype(np.float64)
    assert s[5] == 0 and not q[5].any()
    nz = np.arange(64) != 5
    assert (np.abs(q[nz]).max(1) == 127).all()
    # |x - s q| <= s / 2, plus the binary32 rounding of x / s (at most half an
    # ulp of a quotient below 128, i.e. 2^-18 s: a quotient of 63.4999982 may
    # round to the tie 63.5 and then to 64)
    err = np.abs(xf - oracle.kv_dequant(q, s))
    assert (err[nz] <= s[nz, None].astype(np.float64) * (0.5 + 2.0 ** -17)).all()
    # a row scaled by 2^j keeps its codes and scales its scale by 2^j exactly
    x2 = synth.to_bf16_bits(oracle.bf16_to_f32(x) * np.float32(8.0))
    q3, s3 = oracle.kv_quantize(x2)
    np.testing.assert_array_equal(q3, q)
    np.testing.assert_array_equal(s3, s * np.float32(8.0))


@pytest.mark.parametrize("int8", [True, False])
def test_block_decode_appends_and_attends_the_window(int8):
    r = rng(8 + int8)
    t_max, pos, window = 40, 30, 9
    nq = H * DH
    kv = synth.to_bf16_bits(r.standard_normal((t_max, 2 * DH)).astype(np.float32))
    cache = oracle.kv_cache(t_max, int8)
    oracle.kv_fill(cache, 0, kv[:pos, :DH], kv[:pos, DH:])
    qkv = synth.to_bf16_bits(r.standard_normal(nq + 2 * DH).astype(np.float32))
    out = oracle.attn_block_decode(qkv, cache, pos, window)
    # the new row is cached by the same rule as the others
    if int8:
        qk, sk = oracle.kv_quantize(qkv[None, nq:nq + DH])
        np.testing.assert_array_equal(cache["k"][pos], qk[0])
        assert cache["sk"][pos] == sk[0]
    else:
        np.testing.assert_array_equal(cache["v"][pos], qkv[nq + DH:])
    # the output is the attention over exactly rows pos + 1 - window .. pos
    k, v = oracle.kv_rows(cache, pos + 1 - window, pos + 1)
    q = oracle.bf16_to_f32(qkv[:nq]).astype(np.float64).reshape(H, DH)
    np.testing.assert_array_equal(out, oracle.f64_to_bf16(sdpa(q, k, v, 1 / 16.0).reshape(-1)))
    k1, v1 = oracle.kv_rows(cache, pos - window, pos + 1)     # one row too many
    assert not np.array_equal(out, oracle.f64_to_bf16(sdpa(q, k1, v1, 1 / 16.0).reshape(-1)))


def test_int8_cache_stays_close_to_the_bf16_cache():
    """The INT8 cache changes the attention output by its rounding noise only
    (about 40 dB below the signal for Gaussian rows); a mis-applied scale would
    change it by orders of magnitude."""
    r = rng(11)
    t, nq = 512, H * DH
    kv = synth.to_bf16_bits(r.standard_normal((t, 2 * DH)).astype(np.float32))
    qkv = synth.to_bf16_bits(r.standard_normal(nq + 2 * DH).astype(np.float32) * 2)
    outs = []
    for int8 in (True, False):
        cache = oracle.kv_cache(t, int8)
        oracle.kv_fill(cache, 0, kv[:t - 1, :DH], kv[:t - 1, DH:])
        outs.append(oracle.bf16_to_f32(oracle.attn_block_decode(qkv, cache, t - 1, t)))
    assert oracle.sqnr_db(outs[1], outs[0]) > 30.0


def test_attention_layer_sets():
    assert oracle.attn_precision_map("none").sum() == 0
    assert oracle.attn_precision_map("5+5").sum() == 10
    assert oracle.attn_precision_map("10+10").sum() == 20
    assert oracle.attn_precision_map("all26").sum() == 26
    assert [oracle.attn_window(l, 4096) for l in (0, 1, 6, 25)] == [4096, 1024, 4096, 1024]
