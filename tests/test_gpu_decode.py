"""The persistent decode kernel: at one token, runs of consecutive INT8 FFN
blocks of the stack (Sec. 5's per-layer map) run in one launch with grid-wide
barriers between the gate/up and down phases of every layer.

Bar: bit-identical to the per-launch decode path (the same glue and
quantisation arithmetic, exact int32 sums) for the token stream after every
layer and for the logits, under mixed maps, runs longer than one launch takes,
and the full Gemma-3-1B FFN shapes; the token streams also stay within the
stack's rel-L2 bar of the oracle.  A wait that gives up (forced from the host
with a spin limit of zero polls) must end the kernel and leave a NaN token
stream.  The final glue inside the INT8 lm_head's GEMM must equal the
separate glue launch bit for bit at the full vocabulary.
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


def say(*a):
    print(*a, file=sys.stderr, flush=True)


def dev_bf16(u16):
    return torch.from_numpy(np.ascontiguousarray(u16).view(np.int16)).view(torch.bfloat16).to(DEV)


def dev_f32(a):
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(DEV)


def host_bf16(t):
    return t.detach().cpu().view(torch.int16).numpy().view(np.uint16)


def rel_l2(a, b):
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    return float(np.linalg.norm(a - b) / max(np.linalg.norm(b), 1e-300))


def _stack(cfg, vocab):
    layers_o, i8, bf = [], [], []
    for L in cfg["layers"]:
        qL = oracle.quantize_ffn(L["w_gate"], L["w_up"], L["w_down"], cfg["x_cal"])
        layers_o.append(dict(L, int8=qL))
        i8.append(w8a8.FfnW8A8.from_weights(dev_bf16(L["w_gate"]), dev_bf16(L["w_up"]),
                                            dev_bf16(L["w_down"]), dev_f32(qL["delta_gu"]),
                                            dev_f32(qL["delta_down"])))
        bf.append(w8a8.FfnBF16.from_weights(dev_bf16(L["w_gate"]), dev_bf16(L["w_up"]),
                                            dev_bf16(L["w_down"])))
    d_lm = oracle.smooth_calibrate(cfg["x_cal"], [cfg["w_lm"]])
    return layers_o, w8a8.Stack(i8, bf,
                                w8a8.LinearW8A8.from_weight(dev_bf16(cfg["w_lm"]), dev_f32(d_lm)),
                                w8a8.pack_bf16(dev_bf16(cfg["w_lm"])), vocab)


def _both_paths(stack, x, prec, monkeypatch, lm_head_int8=True):
    """(hidden, logits) from the persistent kernel and from the per-launch path."""
    outs = []
    for flag in ("0", "1"):
        w8a8.set_plan_override("NO_PERSISTENT", int(flag))
        hid, logits = stack.trace(x, prec, lm_head_int8=lm_head_int8, logits=True)
        run = stack.run(x, prec, lm_head_int8)
        outs.append((host_bf16(hid), host_bf16(logits), host_bf16(run)))
    return outs


@pytest.fixture(scope="module")
def small():
    # 34 layers: an all-INT8 map takes two launches (32 + 2 layers)
    cfg = synth.stack_config(m=1, n_layers=34, d=256, f=512, vocab=512)
    return (cfg,) + _stack(cfg, 512)


MAPS_34 = {
    "all": np.ones(34, np.uint8),
    "none": np.zeros(34, np.uint8),
    "mixed": np.array([1, 1, 0, 1, 0, 0, 1, 1, 1] + [1] * 20 + [0, 1, 1, 0, 1], np.uint8),
    "first_bf16": np.array([0] + [1] * 33, np.uint8),
    "last_bf16": np.array([1] * 33 + [0], np.uint8),
}


@pytest.mark.parametrize("name", sorted(MAPS_34))
def test_persistent_bit_identical_to_per_launch(small, name, monkeypatch):
    cfg, _, stack = small
    say("persistent vs per-launch", name)
    prec = MAPS_34[name]
    x = dev_bf16(cfg["x"])
    for lm8 in (True, False):
        (h0, l0, r0), (h1, l1, r1) = _both_paths(stack, x, prec, monkeypatch, lm8)
        np.testing.assert_array_equal(h0, h1)
        np.testing.assert_array_equal(l0, l1)
        np.testing.assert_array_equal(r0, r1)
        np.testing.assert_array_equal(l0, r0)   # trace and plain run agree


def test_persistent_matches_oracle(small, monkeypatch):
    cfg, layers_o, stack = small
    w8a8.set_plan_override("NO_PERSISTENT", 0)
    x = dev_bf16(cfg["x"])
    for name in ("all", "mixed"):
        prec = MAPS_34[name]
        hid = host_bf16(stack.trace(x, prec))
        hid_o = oracle.stack_hidden(cfg["x"], layers_o, prec)
        for l in range(len(prec)):
            err = rel_l2(oracle.bf16_to_f32(hid[l]), oracle.bf16_to_f32(hid_o[l]))
            assert err <= 1e-2, (name, l, err)


@pytest.mark.parametrize("name", ["5+5", "10+10", "all26"])
def test_persistent_full_size_bit_identical(name, monkeypatch):
    say("persistent full size", name)
    cfg = synth.stack_config(m=1, vocab=4096)
    _, stack = _stack(cfg, 4096)
    x = dev_bf16(cfg["x"])
    prec = w8a8.precision_map(name)
    (h0, l0, r0), (h1, l1, r1) = _both_paths(stack, x, prec, monkeypatch)
    np.testing.assert_array_equal(h0, h1)
    np.testing.assert_array_equal(l0, l1)
    np.testing.assert_array_equal(r0, r1)


def test_persistent_failed_wait_gives_nan(small):
    """Force every barrier wait to give up at its first poll: the kernel must
    still end (every wait is bounded), poison its outputs -- the token stream
    after the last layer and the logits of either lm_head are NaN -- and leave
    a record that w8a8_ffn_stack_status reports as ETIMEOUT; the next clean
    call on the same workspace clears it."""
    cfg, _, stack = small
    x = dev_bf16(cfg["x"])
    ws = torch.empty(w8a8.stack_workspace_bytes(1, stack.d, stack.f, stack.vocab),
                     dtype=torch.uint8, device=DEV)
    w8a8.set_plan_override("NO_PERSISTENT", 0)
    w8a8.set_plan_override("DEC_SPIN_LIMIT", 0)
    for name in ("all", "mixed"):
        prec = MAPS_34[name]
        for lm8 in (False, True):
            say("failed wait", name, "lm_head int8" if lm8 else "lm_head bf16")
            hid, logits = stack.trace(x, prec, lm_head_int8=lm8, logits=True, ws=ws)
            assert torch.isnan(hid[-1].float()).all()
            assert torch.isnan(logits.float()).all()
            with pytest.raises(w8a8.W8A8Error) as e:
                w8a8.Stack.status(ws)
            assert e.value.status == w8a8.ETIMEOUT
    w8a8.clear_plan_overrides()
    w8a8.set_plan_override("NO_PERSISTENT", 0)
    hid, logits = stack.trace(x, MAPS_34["all"], lm_head_int8=True, logits=True, ws=ws)
    w8a8.Stack.status(ws)   # clean again
    assert torch.isfinite(hid.float()).all() and torch.isfinite(logits.float()).all()


def test_full_vocab_fused_final_glue_bit_identical(monkeypatch):
    """At one token the final glue (last layer's residual update, final
    RMSNorm and its quantisation) runs inside the INT8 lm_head's streaming
    GEMM; at the full 262144-wide vocabulary (every wave owning its column
    blocks) the logits and the token streams must equal those of the separate
    glue launch bit for bit, after the persistent kernel and after per-launch
    layers alike."""
    say("fused final glue, full vocab")
    cfg = synth.stack_config(m=1, n_layers=2, vocab=512)
    i8, bf = [], []
    for L in cfg["layers"]:
        qL = oracle.quantize_ffn(L["w_gate"], L["w_up"], L["w_down"], cfg["x_cal"])
        i8.append(w8a8.FfnW8A8.from_weights(dev_bf16(L["w_gate"]), dev_bf16(L["w_up"]),
                                            dev_bf16(L["w_down"]), dev_f32(qL["delta_gu"]),
                                            dev_f32(qL["delta_down"])))
        bf.append(w8a8.FfnBF16.from_weights(dev_bf16(L["w_gate"]), dev_bf16(L["w_up"]),
                                            dev_bf16(L["w_down"])))
    g = torch.Generator(device=DEV)
    g.manual_seed(4003)
    vocab = synth.VOCAB
    w_lm = (torch.randn(vocab, synth.D_MODEL, device=DEV, generator=g) * synth.W_SIGMA).to(torch.bfloat16)
    d_lm = (torch.rand(synth.D_MODEL, device=DEV, generator=g) + 0.5).contiguous()
    stack = w8a8.Stack(i8, bf, w8a8.LinearW8A8.from_weight(w_lm, d_lm), w8a8.pack_bf16(w_lm), vocab)
    x = dev_bf16(cfg["x"])
    for persistent in ("0", "1"):
        w8a8.set_plan_override("NO_PERSISTENT", int("1" if persistent == "0" else "0"))
        for prec in (np.array([1, 1], np.uint8), np.array([1, 0], np.uint8), np.array([0, 0], np.uint8)):
            outs = []
            for flag in ("0", "1"):
                w8a8.set_plan_override("NO_FUSED_GLUE", int(flag))
                hid, logits = stack.trace(x, prec, lm_head_int8=True, logits=True)
                outs.append((host_bf16(hid), host_bf16(logits), host_bf16(stack.run(x, prec, True))))
            for a, b in zip(outs[0], outs[1]):
                np.testing.assert_array_equal(a, b)
            assert np.isfinite(oracle.bf16_to_f32(outs[0][1])).all()
