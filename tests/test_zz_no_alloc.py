"""w8a8_ffn_noalloc (the FFN entry point that allocates nothing, its
intermediates in the library's per-GPU scratch array) against w8a8_ffn with a
caller workspace: identical outputs, bit for bit (same kernels), on two
calls in a row, the second with a smaller input, so that what the first call
left in the scratch array cannot leak into the second.  Sizes beyond the
scratch array are refused before any launch."""

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


def host_bf16(t):
    return t.detach().cpu().view(torch.int16).numpy().view(np.uint16)


@pytest.fixture(scope="module")
def layer():
    cfg = synth.ffn_config(m=512)
    q = oracle.quantize_ffn(cfg["w_gate"], cfg["w_up"], cfg["w_down"], cfg["x_cal"][:64])
    f32 = lambda a: torch.from_numpy(np.ascontiguousarray(a, np.float32)).to(DEV)
    L = w8a8.FfnW8A8.from_weights(dev_bf16(cfg["w_gate"]), dev_bf16(cfg["w_up"]),
                                  dev_bf16(cfg["w_down"]), f32(q["delta_gu"]), f32(q["delta_down"]))
    return cfg, L


@pytest.mark.parametrize("sizes", [(512, 5), (128, 1), (300, 37)])
def test_noalloc_ffn_equals_ffn(layer, sizes):
    cfg, L = layer
    for i, m in enumerate(sizes):
        say("ffn_noalloc call %d, m=%d" % (i, m))
        # a different slice of tokens on each call
        x = dev_bf16(np.ascontiguousarray(cfg["x"][i * 7:i * 7 + m]))
        y_ref = host_bf16(w8a8.ffn(L, x))
        y = host_bf16(w8a8.ffn_noalloc(L, x))
        np.testing.assert_array_equal(y, y_ref)


def test_noalloc_ffn_refuses_sizes_beyond_the_scratch(layer):
    cfg, L = layer
    m = 2048
    assert w8a8.ffn_workspace_bytes(m, L.d, L.f) > (32 << 20)
    x = torch.zeros((m, L.d), dtype=torch.bfloat16, device=DEV)
    with pytest.raises(w8a8.W8A8Error) as e:
        w8a8.ffn_noalloc(L, x)
    assert e.value.status == w8a8.EWORKSPACE
    assert b"scratch" in w8a8.lib().w8a8_last_error()
