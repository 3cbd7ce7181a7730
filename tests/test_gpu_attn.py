"""GPU parity of the INT8 key/value cache and the one-token attention over it
(Sec. 4 further speed-ups; Sec. 2 grouped-query layout), and of the attention
projections under the attention layer sets (eq. attnffn55 / attnffn1010 and
the blockwise sets by analogy with eq. ffn55 / ffn1010 / ffnall26).

Bars:
* cache rows (codes and scales): bit-exact against the oracle's per-token
  rule, for rows filled in bulk and for the row each decode step appends;
* attention output (bf16): within one bf16 ulp of the oracle's binary64
  attention rounded once (or, where the output cancels to near zero, within
  2^-16 of the largest output), rel-L2 <= 1e-3.  The kernel forms scores and
  sums in binary32 in another order (products of bf16 queries and INT8 codes
  or bf16 keys are exact; the sums over 256 dimensions and over the rows
  round), so a rounding boundary of the bf16 output can fall between the two
  results;
* INT8 projections: bit-exact (the linear layer's bar); bf16 projections:
  rel-L2 <= 1e-2 (the bf16 path's bar).

The oracle's inputs are drawn by ``synth`` or computed by the oracle; the GPU
is given the same inputs.
"""

import sys

import numpy as np
import pytest
import torch

import oracle
from paper_2608_28003_amd import synth, w8a8

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not torch.cuda.is_available(), reason="needs a GPU")]

DEV = "cuda:0"
DH = 256


def say(*a):
    print(*a, file=sys.stderr, flush=True)


def dev_bf16(u16):
    return torch.from_numpy(np.ascontiguousarray(u16).view(np.int16)).view(torch.bfloat16).to(DEV)


def dev_f32(a):
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(DEV)


def host_bf16(t):
    return t.detach().cpu().view(torch.int16).numpy().view(np.uint16)


def host(t):
    return t.detach().cpu().numpy()


def rel_l2(a, b):
    a = oracle.bf16_to_f32(a).astype(np.float64) if a.dtype == np.uint16 else np.asarray(a, np.float64)
    b = oracle.bf16_to_f32(b).astype(np.float64) if b.dtype == np.uint16 else np.asarray(b, np.float64)
    return float(np.linalg.norm(a - b) / max(np.linalg.norm(b), 1e-300))


def ulp_diff(a, b):
    """Distance in bf16 steps between two bf16 arrays (finite, same sign
    region: the ordered integer images of the bit patterns)."""
    def key(u):
        u = u.astype(np.int32)
        return np.where(u & 0x8000, -(u & 0x7FFF), u)
    return np.abs(key(a) - key(b))


def check_out(out, ref, what):
    """Within one bf16 ulp, or, for outputs that cancel to near zero (where
    the bf16 grid is finer than the binary32 sums resolve), within 2^-16 of
    the largest output magnitude; rel-L2 <= 1e-3."""
    d = ulp_diff(out, ref)
    a = oracle.bf16_to_f32(out).astype(np.float64)
    b = oracle.bf16_to_f32(ref).astype(np.float64)
    near = np.abs(a - b) <= 2.0 ** -16 * np.abs(b).max()
    err = rel_l2(out, ref)
    say("  %s: max %d ulp (%d beyond 1 ulp, all near zero: %s), %.4f bit-identical, rel-L2 %.2e"
        % (what, d.max(), int((d > 1).sum()), bool(near[d > 1].all()), float((d == 0).mean()), err))
    assert ((d <= 1) | near).all(), what
    assert err <= 1e-3, what


def make_caches(inp, t_fill, t_max, int8):
    """The same earlier rows in the oracle's cache and the GPU's, each filled
    by its own side (the GPU quantises through w8a8_kv_quantize)."""
    oc = oracle.kv_cache(t_max, int8)
    oracle.kv_fill(oc, 0, inp["k"][:t_fill], inp["v"][:t_fill])
    gc = w8a8.KVCache(t_max, int8, DEV)
    if t_fill:
        gc.fill(0, dev_bf16(inp["k"][:t_fill]), dev_bf16(inp["v"][:t_fill]))
    return oc, gc


def test_kv_quantize_bit_exact_with_stride_and_edge_rows():
    """Rows read with the stride of a fused QKV output (the key columns of
    [q | k | v] rows), plus a zero row, a row of one nonzero value, ties at
    x / s = k + 1/2 and subnormal-range values."""
    rng = np.random.default_rng(5)
    m, width = 300, 4 * DH + 2 * DH
    qkv = (rng.standard_normal((m, width)) * 2).astype(np.float32)
    qkv[7, 4 * DH:5 * DH] = 0
    qkv[8, 4 * DH:5 * DH] = 0
    qkv[8, 4 * DH + 3] = -3.5
    qkv[9, 4 * DH:5 * DH] = np.arange(DH, dtype=np.float32) - 127.0   # s = 1: ties .. exact
    qkv[10, 4 * DH:5 * DH] = 2.5 * (np.arange(DH) % 5 - 2)             # s = 5/127
    qkv[11, 4 * DH:5 * DH] *= np.float32(1e-38)
    x = synth.to_bf16_bits(qkv)
    codes, scales = w8a8.kv_quantize(dev_bf16(x)[:, 4 * DH:5 * DH])
    q_o, s_o = oracle.kv_quantize(x[:, 4 * DH:5 * DH])
    np.testing.assert_array_equal(host(codes), q_o)
    np.testing.assert_array_equal(host(scales), s_o)


CASES = [  # t_max, pos, window: one row, one pass, a pass and a row, ragged, sliding, many workgroups
    (1, 0, 4096), (64, 63, 4096), (65, 64, 4096), (300, 299, 4096),
    (2000, 1999, 1024), (5000, 4321, 4096), (32768, 32767, 32768)]


@pytest.mark.parametrize("int8", [True, False])
@pytest.mark.parametrize("t_max,pos,window", CASES)
def test_attn_decode_matches_oracle(int8, t_max, pos, window):
    say("attn decode int8=%d t_max=%d pos=%d window=%d" % (int8, t_max, pos, window))
    inp = synth.kv_decode_inputs(5100 + pos, pos, n_heads=4)
    oc, gc = make_caches(inp, pos, t_max, int8)
    out_o = oracle.attn_block_decode(inp["qkv"], oc, pos, window)
    out = w8a8.attn_decode(dev_bf16(inp["qkv"]), gc, pos, window)
    torch.cuda.synchronize()
    if int8:  # every row the attention read, and the appended one
        np.testing.assert_array_equal(host(gc.k[:pos + 1]), oc["k"][:pos + 1])
        np.testing.assert_array_equal(host(gc.sk[:pos + 1]), oc["sk"][:pos + 1])
        np.testing.assert_array_equal(host(gc.v[:pos + 1]), oc["v"][:pos + 1])
        np.testing.assert_array_equal(host(gc.sv[:pos + 1]), oc["sv"][:pos + 1])
    else:
        np.testing.assert_array_equal(host_bf16(gc.k[pos]), oc["k"][pos])
        np.testing.assert_array_equal(host_bf16(gc.v[pos]), oc["v"][pos])
    check_out(host_bf16(out), out_o, "out")


@pytest.mark.parametrize("n_heads", [1, 2, 8])
def test_attn_decode_head_counts(n_heads):
    t_max, pos, window = 700, 650, 4096
    inp = synth.kv_decode_inputs(5200 + n_heads, pos, n_heads=n_heads)
    oc, gc = make_caches(inp, pos, t_max, True)
    out_o = oracle.attn_block_decode(inp["qkv"], oc, pos, window, n_heads=n_heads)
    out = w8a8.attn_decode(dev_bf16(inp["qkv"]), gc, pos, window, n_heads=n_heads)
    check_out(host_bf16(out), out_o, "heads %d" % n_heads)


@pytest.mark.timeout(300)
def test_attn_decode_long_context_several_passes_per_workgroup():
    """131072 rows: 2048 passes of 64 over 256 workgroups, so every workgroup
    carries its running maximum and sum across eight passes."""
    t_max = pos = 131071
    inp = synth.kv_decode_inputs(5300, pos, n_heads=4)
    oc, gc = make_caches(inp, pos, t_max + 1, True)
    out_o = oracle.attn_block_decode(inp["qkv"], oc, pos, t_max + 1)
    out = w8a8.attn_decode(dev_bf16(inp["qkv"]), gc, pos, t_max + 1)
    check_out(host_bf16(out), out_o, "131072 rows")


@pytest.mark.parametrize("int8", [True, False])
def test_consecutive_decode_steps(int8):
    """Five steps in a row on one cache, each appending its token: the cache
    the kernel wrote is read back by the next step (sliding window 64)."""
    t_max, p0, window = 200, 120, 64
    inp = synth.kv_decode_inputs(5400, p0, n_heads=4)
    oc, gc = make_caches(inp, p0, t_max, int8)
    for step in range(5):
        row = synth.kv_decode_inputs(5500 + step, 0, n_heads=4)["qkv"]
        out_o = oracle.attn_block_decode(row, oc, p0 + step, window)
        out = w8a8.attn_decode(dev_bf16(row), gc, p0 + step, window)
        check_out(host_bf16(out), out_o, "step %d" % step)
    if int8:
        np.testing.assert_array_equal(host(gc.k[:p0 + 5]), oc["k"][:p0 + 5])
        np.testing.assert_array_equal(host(gc.sv[:p0 + 5]), oc["sv"][:p0 + 5])


def _attn_layers(n_layers, seed=5600):
    """Per layer: fused QKV and O weights (bf16), their INT8 codes from the
    oracle's calibration, the synthetic block input and attention output."""
    cfg = synth.attn_config(m=1, seed_base=seed)
    layers = []
    for l in range(n_layers):
        c = synth.attn_config(m=1, seed_base=seed + 10 * (l + 1))
        d_qkv = oracle.smooth_calibrate(c["x_cal"], [c["w_qkv"]])
        d_o = oracle.smooth_calibrate(c["x_o"], [c["w_o"]])
        wq_qkv, s_qkv = oracle.quantize_weights(c["w_qkv"], d_qkv)
        wq_o, s_o = oracle.quantize_weights(c["w_o"], d_o)
        layers.append(dict(w_qkv=c["w_qkv"], w_o=c["w_o"], wq_qkv=wq_qkv, s_qkv=s_qkv,
                           delta_qkv=d_qkv, wq_o=wq_o, s_o=s_o, delta_o=d_o, x=c["x"], x_o=c["x_o"]))
    return cfg, layers


@pytest.mark.parametrize("name", ["5+5", "all26"])
def test_attention_projection_map_with_int8_cache(name):
    """26 attention blocks at one token under an attention layer set: each
    layer's QKV projection (INT8 in the set, bf16 outside), the INT8-cache
    attention of that projection's row over its own cache (global layers the
    whole 600-token context, the others the sliding window, here 256 so both
    kinds differ), and the O projection of the attention output."""
    prec = oracle.attn_precision_map(name)
    n_layers, ctx, window = len(prec), 600, 256
    _, layers = _attn_layers(n_layers)
    for l, L in enumerate(layers):
        int8 = bool(prec[l])
        qkv_o, _ = oracle.attn_block_proj_decode(L["x"], L["x_o"], L, int8)
        x = dev_bf16(L["x"])
        n_qkv, n_o = L["w_qkv"].shape[0], L["w_o"].shape[0]
        if int8:
            lin_qkv = w8a8.LinearW8A8.from_weight(dev_bf16(L["w_qkv"]), dev_f32(L["delta_qkv"]))
            qkv = w8a8.linear(lin_qkv, x, out_dtype=torch.bfloat16)
            np.testing.assert_array_equal(host_bf16(qkv), qkv_o, err_msg="qkv layer %d" % l)
        else:
            qkv = w8a8.bf16_linear(x, w8a8.pack_bf16(dev_bf16(L["w_qkv"])), n_qkv, L["w_qkv"].shape[1])
            assert rel_l2(host_bf16(qkv), qkv_o) <= 1e-2, l
        # attention from the oracle's projection row, over this layer's cache
        inp = synth.kv_decode_inputs(5700 + l, ctx - 1)
        win = window if l not in oracle.GLOBAL_LAYERS else ctx
        oc, gc = make_caches(inp, ctx - 1, ctx, True)
        att_o = oracle.attn_block_decode(qkv_o.reshape(-1), oc, ctx - 1, win)
        att = w8a8.attn_decode(dev_bf16(qkv_o.reshape(-1)), gc, ctx - 1, win)
        check_out(host_bf16(att), att_o, "layer %d attention" % l)
        # O projection of the oracle's attention output
        _, o_o = oracle.attn_block_proj_decode(L["x"], att_o[None, :], L, int8)
        if int8:
            lin_o = w8a8.LinearW8A8.from_weight(dev_bf16(L["w_o"]), dev_f32(L["delta_o"]))
            o = w8a8.linear(lin_o, dev_bf16(att_o[None, :]), out_dtype=torch.bfloat16)
            np.testing.assert_array_equal(host_bf16(o), o_o, err_msg="o layer %d" % l)
        else:
            o = w8a8.bf16_linear(dev_bf16(att_o[None, :]), w8a8.pack_bf16(dev_bf16(L["w_o"])), n_o, 1024)
            assert rel_l2(host_bf16(o), o_o) <= 1e-2, l


@pytest.mark.parametrize("int8", [True, False])
@pytest.mark.parametrize("t_max,pos,window", [(200, 150, 1), (200, 150, 2), (5000, 100, 4096), (4097, 4096, 4097)])
def test_attn_decode_edge_windows(int8, t_max, pos, window):
    """A window of one row (the output is the new value alone), of two, a
    cache far longer than the rows written, and a pass boundary right before
    the new row with many workgroups."""
    say("attn edge int8=%d t_max=%d pos=%d window=%d" % (int8, t_max, pos, window))
    inp = synth.kv_decode_inputs(6100 + pos + window, pos, n_heads=4)
    oc, gc = make_caches(inp, pos, t_max, int8)
    out_o = oracle.attn_block_decode(inp["qkv"], oc, pos, window)
    out = w8a8.attn_decode(dev_bf16(inp["qkv"]), gc, pos, window)
    check_out(host_bf16(out), out_o, "edge")
    if window == 1:  # softmax over one row: the value itself, for every head
        v = oracle.kv_rows(oc, pos, pos + 1)[1][0]
        np.testing.assert_array_equal(out_o, oracle.f64_to_bf16(np.tile(v, 4)))


def test_attn_decode_eight_heads_bf16_cache():
    t_max, pos, window = 3000, 2999, 3000
    inp = synth.kv_decode_inputs(6200, pos, n_heads=8)
    oc, gc = make_caches(inp, pos, t_max, False)
    out_o = oracle.attn_block_decode(inp["qkv"], oc, pos, window, n_heads=8)
    out = w8a8.attn_decode(dev_bf16(inp["qkv"]), gc, pos, window, n_heads=8)
    check_out(host_bf16(out), out_o, "8 heads bf16")
