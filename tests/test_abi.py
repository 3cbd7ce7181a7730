"""C-ABI checks that need no GPU: the library loads, exports every symbol the
header declares, and rejects bad arguments on the host before any HIP call.
Every call below fails validation, so no kernel is ever launched."""

import ctypes
import os
import re

import numpy as np
import pytest

from paper_2608_28003_amd import w8a8
import oracle

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "w8a8.h")

P = ctypes.c_void_p
FAKE = P(0x1000)          # aligned, never dereferenced: validation fails first
MISALIGNED = P(0x1004)


def _declared(header=HEADER):
    text = open(header).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(w8a8_[a-z0-9_]+)\s*\(", text)))


def test_library_exports_every_declared_symbol():
    L = w8a8.lib()
    names = _declared()
    assert len(names) >= 25
    for n in names:
        assert hasattr(L, n), n
    assert set(names) == set(w8a8.exported_names())


def test_peak_library_exports_its_header_and_rejects_bad_arguments():
    """The benchmark's ceiling probes (include/w8a8_peak.h): every declared
    symbol is exported, and bad arguments return 1 before any launch."""
    from paper_2608_28003_amd import build as hip_build
    L = ctypes.CDLL(hip_build.PEAK_LIB_PATH)
    names = _declared(os.path.join(ROOT, "include", "w8a8_peak.h"))
    assert len(names) == 4
    for n in names:
        assert hasattr(L, n), n
    L.w8a8_peak_read_write.argtypes = [P, ctypes.c_int64, ctypes.c_int, P, ctypes.c_int,
                                       ctypes.c_int, P, P]
    L.w8a8_peak_read.argtypes = [P, ctypes.c_size_t, ctypes.c_int, P, P]
    assert L.w8a8_peak_read_write(FAKE, 262144, 1100, FAKE, 64, 1024, FAKE, None) == 1  # k % 64
    assert L.w8a8_peak_read_write(FAKE, 262144, 1600, FAKE, 64, 1024, FAKE, None) == 1  # k > 1536
    assert L.w8a8_peak_read_write(FAKE, 100, 1152, FAKE, 64, 1024, FAKE, None) == 1     # n % 64
    assert L.w8a8_peak_read_write(MISALIGNED, 262144, 1152, FAKE, 64, 1024, FAKE, None) == 1
    assert L.w8a8_peak_read_write(FAKE, 262144, 1152, None, 64, 1024, FAKE, None) == 1
    assert L.w8a8_peak_read(FAKE, 8, 16, FAKE, None) == 1


def test_status_strings():
    L = w8a8.lib()
    for code in range(6):
        assert L.w8a8_status_str(code) != b"unknown status"
    assert L.w8a8_status_str(99) == b"unknown status"


def test_packed_sizes():
    assert w8a8.packed_bytes(6912, 1152) == 6912 * 1152
    assert w8a8.packed_bytes(262144, 1152) == 301989888
    assert w8a8.packed_bytes(1, 16) == 16 * 64          # padded to a 16 x 64 fragment
    assert w8a8.packed_bytes(17, 65) == 32 * 128
    assert w8a8.packed_bytes(0, 16) == 0
    assert w8a8.packed_bf16_bytes(6912, 1152) == 6912 * 1152 * 2
    assert w8a8.packed_bf16_bytes(3, 40) == 16 * 64 * 2


def test_workspace_queries_cover_buffers():
    m, d, f = 128, 1152, 6912
    ws = w8a8.ffn_workspace_bytes(m, d, f)
    assert ws >= w8a8.packed_bytes(m, d) + m * 4 + m * f * 2 + w8a8.packed_bytes(m, f) + m * 4
    assert w8a8.linear_workspace_bytes(1, 262144, 1152) >= w8a8.packed_bytes(1, 1152) + 4
    assert w8a8.stack_workspace_bytes(512, d, f, 262144) > w8a8.ffn_workspace_bytes(512, d, f)
    assert w8a8.linear_workspace_bytes(0, 1, 1) == 0


def test_precision_maps_from_library_match_oracle():
    for name in ("bf16", "5+5", "10+10", "all26"):
        np.testing.assert_array_equal(w8a8.precision_map(name), oracle.precision_map(name))
    with pytest.raises(ValueError):
        w8a8.precision_map("3+3")
    with pytest.raises(ValueError):
        w8a8.precision_map("5+5", 20)


def _status(fn, *args):
    return fn(*args)


def test_quantize_act_validation():
    L = w8a8.lib()
    q = L.w8a8_quantize_act
    assert q(None, w8a8.BF16, 4, 1152, None, FAKE, FAKE, None) == w8a8.EINVAL
    assert q(FAKE, w8a8.BF16, 0, 1152, None, FAKE, FAKE, None) == w8a8.EINVAL
    assert q(FAKE, w8a8.BF16, 4, 1000, None, FAKE, FAKE, None) == w8a8.EUNSUPPORTED
    assert q(FAKE, w8a8.BF16, 4, w8a8.MAX_K + 16, None, FAKE, FAKE, None) == w8a8.EUNSUPPORTED
    assert q(FAKE, 7, 4, 1152, None, FAKE, FAKE, None) == w8a8.EUNSUPPORTED
    assert q(MISALIGNED, w8a8.BF16, 4, 1152, None, FAKE, FAKE, None) == w8a8.EINVAL
    assert b"aligned" in L.w8a8_last_error()


def test_quantize_weights_and_calibration_validation():
    L = w8a8.lib()
    assert L.w8a8_quantize_weights(FAKE, w8a8.F32, 16, 24, None, FAKE, FAKE, None) == w8a8.EUNSUPPORTED
    assert L.w8a8_quantize_weights(FAKE, w8a8.F32, 0, 64, None, FAKE, FAKE, None) == w8a8.EINVAL
    assert L.w8a8_quantize_weights(FAKE, w8a8.F32, 16, 64, MISALIGNED, FAKE, FAKE, None) == w8a8.EINVAL
    assert L.w8a8_smooth_delta(FAKE, FAKE, 64, 1.5, FAKE, None) == w8a8.EUNSUPPORTED
    assert L.w8a8_smooth_delta(FAKE, None, 64, 0.5, FAKE, None) == w8a8.EINVAL
    ws = (P * 2)(FAKE.value, FAKE.value)
    rows = (ctypes.c_int64 * 2)(6912, 6912)
    sc = L.w8a8_smooth_calibrate
    assert sc(FAKE, ws, rows, 2, w8a8.BF16, 1152, 1.5, FAKE, None) == w8a8.EUNSUPPORTED
    assert sc(FAKE, ws, rows, 2, 9, 1152, 0.5, FAKE, None) == w8a8.EUNSUPPORTED
    assert sc(FAKE, ws, rows, 0, w8a8.BF16, 1152, 0.5, FAKE, None) == w8a8.EINVAL
    assert sc(FAKE, None, rows, 2, w8a8.BF16, 1152, 0.5, FAKE, None) == w8a8.EINVAL
    assert sc(None, ws, rows, 2, w8a8.BF16, 1152, 0.5, FAKE, None) == w8a8.EINVAL
    bad = (P * 2)(FAKE.value, None)
    assert sc(FAKE, bad, rows, 2, w8a8.BF16, 1152, 0.5, FAKE, None) == w8a8.EINVAL
    zero = (ctypes.c_int64 * 2)(6912, 0)
    assert sc(FAKE, ws, zero, 2, w8a8.BF16, 1152, 0.5, FAKE, None) == w8a8.EINVAL
    assert L.w8a8_col_absmax(FAKE, w8a8.BF16, 0, 64, FAKE, None) == w8a8.EINVAL
    assert L.w8a8_pack_bf16(FAKE, 16, 48, FAKE, None) == w8a8.EUNSUPPORTED


def test_linear_and_ffn_validation():
    L = w8a8.lib()
    d = w8a8.LinearDesc(6912, 1152, FAKE, FAKE, None)
    need = w8a8.linear_workspace_bytes(16, 6912, 1152)
    assert L.w8a8_linear(ctypes.byref(d), FAKE, w8a8.F32, 16, FAKE, w8a8.F32, FAKE, need - 1, None) == w8a8.EWORKSPACE
    assert L.w8a8_linear(None, FAKE, w8a8.F32, 16, FAKE, w8a8.F32, FAKE, need, None) == w8a8.EINVAL
    assert L.w8a8_linear(ctypes.byref(d), FAKE, w8a8.F32, 16, FAKE, 5, FAKE, need, None) == w8a8.EUNSUPPORTED
    bad = w8a8.LinearDesc(6912, 1100, FAKE, FAKE, None)
    assert L.w8a8_linear(ctypes.byref(bad), FAKE, w8a8.F32, 16, FAKE, w8a8.F32, FAKE, need, None) == w8a8.EUNSUPPORTED
    nul = w8a8.LinearDesc(6912, 1152, None, FAKE, None)
    assert L.w8a8_linear(ctypes.byref(nul), FAKE, w8a8.F32, 16, FAKE, w8a8.F32, FAKE, need, None) == w8a8.EINVAL
    f = w8a8.FfnDesc(1152, 6912, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE)
    need = w8a8.ffn_workspace_bytes(8, 1152, 6912)
    assert L.w8a8_ffn(ctypes.byref(f), FAKE, 8, FAKE, FAKE, need - 1, None) == w8a8.EWORKSPACE
    f2 = w8a8.FfnDesc(1152, 6912, FAKE, FAKE, None, FAKE, FAKE, FAKE, FAKE, FAKE)
    assert L.w8a8_ffn(ctypes.byref(f2), FAKE, 8, FAKE, FAKE, need, None) == w8a8.EINVAL
    assert L.w8a8_lm_head(ctypes.byref(d), FAKE, 0, FAKE, FAKE, 1 << 30, None) == w8a8.EINVAL
    assert L.w8a8_gemm_i8_i32(FAKE, 4, FAKE, 16, 1000, FAKE, FAKE, 1 << 20, None) == w8a8.EUNSUPPORTED
    assert L.w8a8_bf16_linear(FAKE, 4, FAKE, 16, 48, FAKE, None, 0, None) == w8a8.EUNSUPPORTED


def test_geglu_requant_validation():
    L = w8a8.lib()
    g = L.w8a8_geglu_requant
    assert g(None, FAKE, 4, 6912, None, FAKE, FAKE, None, None) == w8a8.EINVAL
    assert g(FAKE, FAKE, 0, 6912, None, FAKE, FAKE, None, None) == w8a8.EINVAL
    assert g(FAKE, FAKE, 4, 6904, None, FAKE, FAKE, None, None) == w8a8.EUNSUPPORTED
    assert g(FAKE, FAKE, 4, w8a8.MAX_K + 16, None, FAKE, FAKE, None, None) == w8a8.EUNSUPPORTED
    assert g(FAKE, FAKE, 4, 6912, MISALIGNED, FAKE, FAKE, None, None) == w8a8.EINVAL
    assert g(FAKE, FAKE, 4, 6912, None, FAKE, FAKE, MISALIGNED, None) == w8a8.EINVAL


def test_kv_cache_and_attention_validation():
    L = w8a8.lib()
    q = L.w8a8_kv_quantize
    assert q(None, 4, 256, FAKE, FAKE, None) == w8a8.EINVAL
    assert q(FAKE, 0, 256, FAKE, FAKE, None) == w8a8.EINVAL
    assert q(FAKE, 4, 255, FAKE, FAKE, None) == w8a8.EINVAL
    assert q(FAKE, 4, 260, FAKE, FAKE, None) == w8a8.EINVAL
    assert q(FAKE, 4, 256, MISALIGNED, FAKE, None) == w8a8.EINVAL
    assert L.w8a8_attn_decode_workspace_bytes(64) == 0
    assert L.w8a8_attn_decode_workspace_bytes(32768) > 0
    a = L.w8a8_attn_decode
    ok = (FAKE, 4, 10, 1024, FAKE, FAKE, FAKE, FAKE, 64, FAKE, None, 0, None)
    for i, bad, code in ((0, None, w8a8.EINVAL), (1, 3, w8a8.EUNSUPPORTED), (1, 16, w8a8.EUNSUPPORTED),
                         (2, 64, w8a8.EINVAL), (2, -1, w8a8.EINVAL), (3, 0, w8a8.EINVAL),
                         (4, None, w8a8.EINVAL), (5, MISALIGNED, w8a8.EINVAL),
                         (8, 0, w8a8.EINVAL), (9, None, w8a8.EINVAL)):
        args = list(ok)
        args[i] = bad
        assert a(*args) == code, (i, bad)
    # a long context needs the workspace
    assert a(FAKE, 4, 32767, 32768, FAKE, FAKE, FAKE, FAKE, 32768, FAKE, None, 0, None) == w8a8.EINVAL
    assert a(FAKE, 4, 32767, 32768, FAKE, FAKE, FAKE, FAKE, 32768, FAKE, FAKE, 64, None) == w8a8.EWORKSPACE
    b = L.w8a8_attn_decode_bf16
    assert b(FAKE, 4, 10, 1024, None, FAKE, 64, FAKE, None, 0, None) == w8a8.EINVAL
    assert b(FAKE, 5, 10, 1024, FAKE, FAKE, 64, FAKE, None, 0, None) == w8a8.EUNSUPPORTED


def test_stack_status_validation_and_codes():
    L = w8a8.lib()
    assert L.w8a8_ffn_stack_status(None, 1 << 20, None) == w8a8.EINVAL
    assert L.w8a8_ffn_stack_status(FAKE, 16, None) == w8a8.EWORKSPACE
    assert b"persistent" in L.w8a8_status_str(w8a8.ETIMEOUT)


def test_plan_overrides_are_explicit():
    """The planner reads overrides set through the ABI, never the environment."""
    L = w8a8.lib()
    assert L.w8a8_set_plan_override(b"NOT_A_KNOB", 1) == -1
    assert L.w8a8_set_plan_override(None, 1) == -1
    for name in (b"GLU_TILE", b"GEMM_SPLITS", b"NO_PERSISTENT", b"DEC_SPIN_LIMIT"):
        assert L.w8a8_set_plan_override(name, 1) == 0
    L.w8a8_clear_plan_overrides()
    with pytest.raises(ValueError):
        w8a8.set_plan_override("W8A8_GLU_TILE", 3)
    src = open(os.path.join(ROOT, "paper_2608_28003_amd", "csrc", "api.hip")).read()
    assert "getenv" not in src


def test_stack_validation():
    L = w8a8.lib()
    i8 = (w8a8.FfnDesc * 2)()
    bf = (w8a8.Bf16FfnDesc * 2)(w8a8.Bf16FfnDesc(1152, 6912, FAKE, FAKE, FAKE),
                                w8a8.Bf16FfnDesc(1152, 6912, FAKE, FAKE, FAKE))
    sd = w8a8.StackDesc(2, 1152, 6912, 4096, i8, bf, w8a8.LinearDesc(), FAKE)
    need = w8a8.stack_workspace_bytes(4, 1152, 6912, 4096)
    prec = np.array([1, 0], np.uint8)   # layer 0 asks for INT8 but has no descriptor
    assert L.w8a8_ffn_stack(ctypes.byref(sd), prec.ctypes.data_as(P), 0, FAKE, 4, FAKE, FAKE,
                            need, None) == w8a8.EINVAL
    prec = np.array([0, 0], np.uint8)
    assert L.w8a8_ffn_stack(ctypes.byref(sd), prec.ctypes.data_as(P), 1, FAKE, 4, FAKE, FAKE,
                            need, None) == w8a8.EINVAL   # lm_head INT8 requested, desc empty
    assert L.w8a8_ffn_stack(ctypes.byref(sd), prec.ctypes.data_as(P), 0, FAKE, 4, FAKE, FAKE,
                            need - 1, None) == w8a8.EWORKSPACE


def test_fragment_layout_helpers_roundtrip():
    rng = np.random.default_rng(3)
    for rows, k in [(1, 16), (17, 80), (48, 1152), (5, 64)]:
        q = rng.integers(-127, 128, (rows, k), dtype=np.int8)
        packed = w8a8.rowmajor_to_frag(q)
        assert packed.size == w8a8.packed_bytes(rows, k)
        np.testing.assert_array_equal(w8a8.frag_to_rowmajor(packed, rows, k), q)
    # lane l of fragment (0, 0) holds row l % 16, columns (l // 16) * 16 .. +15
    q = np.arange(16 * 64, dtype=np.int64).reshape(16, 64)
    qq = (q % 251 - 125).astype(np.int8)
    packed = w8a8.rowmajor_to_frag(qq).view(np.int8)
    for lane in (0, 5, 16, 37, 63):
        r, g = lane % 16, lane // 16
        np.testing.assert_array_equal(packed[16 * lane:16 * lane + 16], qq[r, 16 * g:16 * g + 16])
