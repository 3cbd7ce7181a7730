"""AddressSanitizer and UndefinedBehaviorSanitizer builds of the host code, on
the CPU: the oracle's C loops, and the library's host layer (argument
validation, workspace sizing, the GEMM planner, precision maps, layer ranking,
status strings), which runs before any HIP call.  Each is compiled with the
sanitizers into a temporary directory and exercised in a child process that
preloads the matching sanitizer runtime; any report fails the test.

GPU code is never instrumented here: on the hipcc line every sanitizer flag
is passed to the host compilation only.
"""

import os
import subprocess
import sys
import textwrap

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

SAN_MARKERS = ("ERROR: AddressSanitizer", "runtime error:", "ERROR: LeakSanitizer",
               "UndefinedBehaviorSanitizer")


def _have(cmd):
    try:
        return subprocess.run(cmd, capture_output=True).returncode == 0
    except OSError:
        return False


def _run_child(code, env_extra, timeout=600):
    env = dict(os.environ)
    env.update(env_extra)
    env["ASAN_OPTIONS"] = "detect_leaks=0:abort_on_error=0:halt_on_error=1"
    env["UBSAN_OPTIONS"] = "print_stacktrace=1:halt_on_error=1"
    r = subprocess.run([sys.executable, "-c", code], capture_output=True, text=True, env=env,
                       cwd=ROOT, timeout=timeout)
    out = r.stdout + r.stderr
    for marker in SAN_MARKERS:
        assert marker not in out, out[-4000:]
    assert r.returncode == 0, out[-4000:]
    return out


@pytest.mark.timeout(600)
@pytest.mark.skipif(not _have(["gcc", "--version"]), reason="needs gcc")
def test_oracle_under_address_and_undefined_behaviour_sanitizers(tmp_path):
    src = os.path.join(ROOT, "oracle", "w8a8_oracle.c")
    lib = str(tmp_path / "liborc_san.so")
    subprocess.run(["gcc", "-O1", "-g", "-std=c11", "-fPIC", "-shared", "-fopenmp",
                    "-ffp-contract=off", "-fno-omit-frame-pointer",
                    "-fsanitize=address,undefined", "-fno-sanitize-recover=undefined",
                    "-o", lib, src, "-lm"], check=True)
    asan = subprocess.run(["gcc", "-print-file-name=libasan.so"], capture_output=True,
                          text=True).stdout.strip()
    code = textwrap.dedent("""
        import numpy as np
        import oracle
        from paper_2608_28003_amd import synth
        rng = np.random.default_rng(1)
        for m, k in ((1, 16), (3, 64), (17, 1152), (5, 100)):
            x = synth.to_bf16_bits(rng.standard_normal((m, k)).astype(np.float32) * 3)
            x[0] = 0
            d = (rng.random(k) + 0.5).astype(np.float32)
            q, s = oracle.quantize_act(x, d)
            qw, sw = oracle.quantize_weights(x, d)
            acc = oracle.gemm_i32(q, qw)
            y = oracle.dequant(acc, s, sw)
            oracle.smooth_calibrate(x, [x])
            oracle.linear_f64(x, x)
            oracle.rmsnorm(x)
            oracle.geglu(y, y)
            qf, sf = oracle.quantize_act_fp8(x, d)
            oracle.dequant_fp8(oracle.gemm_fp8(qf, qf), sf, sf)
            oracle.kv_quantize(synth.to_bf16_bits(rng.standard_normal((m, 256)).astype(np.float32)))
        cfg = synth.ffn_config(m=4, d=64, f=128)
        qf = oracle.quantize_ffn(cfg["w_gate"], cfg["w_up"], cfg["w_down"], cfg["x_cal"][:16])
        oracle.w8a8_ffn(cfg["x"], qf, stages=True)
        oracle.bf16_ffn(cfg["x"], cfg["w_gate"], cfg["w_up"], cfg["w_down"])
        for t in (1, 2, 65):
            q = rng.standard_normal((4, 256)); kk = rng.standard_normal((t, 256))
            oracle.attn_decode(q, kk, kk)
        c = oracle.kv_cache(8, True)
        row = synth.to_bf16_bits(rng.standard_normal(1536).astype(np.float32))
        oracle.attn_block_decode(row, c, 0, 8)
        oracle.attn_block_decode(row, c, 1, 1)
        print("oracle ok")
    """)
    out = _run_child(code, {"LD_PRELOAD": asan, "W8A8_ORACLE_LIB": lib})
    assert "oracle ok" in out


def _clang_asan_runtime():
    import glob
    c = sorted(glob.glob("/opt/rocm/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so"))
    return c[-1] if c else None


@pytest.mark.timeout(900)
@pytest.mark.skipif(not os.path.exists("/opt/rocm/bin/hipcc") or _clang_asan_runtime() is None,
                    reason="needs hipcc and clang's sanitizer runtime")
def test_host_layer_under_address_and_undefined_behaviour_sanitizers(tmp_path):
    """The C ABI's host code (api.hip) rebuilt with host-only sanitizers and
    linked with the other translation units; every call below returns before
    touching a device."""
    from paper_2608_28003_amd import build as hip_build
    csrc = hip_build.CSRC
    objs = []
    for src in sorted(os.listdir(csrc)):
        if not src.endswith(".hip"):
            continue
        path = os.path.join(csrc, src)
        # the other translation units as the last build left them, when that
        # build is newer than every source (they hold no host validation code)
        built = os.path.join(hip_build.BUILD_DIR, src + ".o")
        newest = max(os.path.getmtime(os.path.join(csrc, f)) for f in os.listdir(csrc)
                     if f.endswith((".hip", ".h")))
        if src != "api.hip" and os.path.exists(built) and os.path.getmtime(built) >= newest:
            objs.append(built)
            continue
        obj = str(tmp_path / (src + ".o"))
        cmd = ["/opt/rocm/bin/hipcc"] + hip_build.CFLAGS + ["-g", "-c", path, "-o", obj]
        if src == "api.hip":
            cmd += ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
                    "-Xarch_host", "-fno-sanitize-recover=undefined",
                    "-Xarch_host", "-fno-omit-frame-pointer"]
        r = subprocess.run(cmd, capture_output=True, text=True)
        assert r.returncode == 0, r.stderr[-3000:]
        objs.append(obj)
    lib = str(tmp_path / "libw8a8_san.so")
    r = subprocess.run(["/opt/rocm/bin/hipcc", "--offload-arch=" + hip_build.ARCH, "-shared", "-fPIC",
                        "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
                        "-shared-libasan", "-o", lib] + objs, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-3000:]
    code = textwrap.dedent("""
        import ctypes
        import numpy as np
        from paper_2608_28003_amd import w8a8
        w8a8.LIB_PATH = %r
        L = w8a8.lib()
        FAKE = ctypes.c_void_p(1 << 20)
        MIS = ctypes.c_void_p((1 << 20) + 4)
        for m in (1, 2, 7, 16, 17, 33, 64, 65, 128, 300, 512, 1024, 2048, 4096):
            for n, k in ((6912, 1152), (1152, 6912), (1536, 1152), (1152, 1024), (262144, 1152)):
                L.w8a8_linear_workspace_bytes(m, n, k)
                L.w8a8_lm_head_workspace_bytes(m, n, k)
                L.w8a8_bf16_linear_workspace_bytes(m, n, k)
                L.w8a8_fp8_linear_workspace_bytes(m, n, k)
            L.w8a8_ffn_workspace_bytes(m, 1152, 6912)
            L.w8a8_bf16_ffn_workspace_bytes(m, 1152, 6912)
            L.w8a8_fp8_ffn_workspace_bytes(m, 1152, 6912)
            L.w8a8_stack_workspace_bytes(m, 1152, 6912, 262144)
            L.w8a8_stack_sensitivity_workspace_bytes(m, 1152, 6912, 262144, 26)
        for t in (1, 64, 65, 4096, 65536, 131072):
            L.w8a8_attn_decode_workspace_bytes(t)
        for n, k in ((1, 16), (262144, 1152), (17, 6912)):
            L.w8a8_packed_bytes(n, k)
            L.w8a8_packed_bf16_bytes(n, k)
        # validation failures: every one returns a status and sets the message
        assert L.w8a8_quantize_act(None, 1, 4, 1152, None, FAKE, FAKE, None) == w8a8.EINVAL
        assert L.w8a8_quantize_act(FAKE, 1, 4, 1100, None, FAKE, FAKE, None) == w8a8.EUNSUPPORTED
        assert L.w8a8_quantize_act(MIS, 1, 4, 1152, None, FAKE, FAKE, None) == w8a8.EINVAL
        assert len(L.w8a8_last_error()) > 0
        assert L.w8a8_geglu_requant(FAKE, FAKE, 0, 6912, None, FAKE, FAKE, None, None) == w8a8.EINVAL
        assert L.w8a8_kv_quantize(FAKE, 4, 255, FAKE, FAKE, None) == w8a8.EINVAL
        assert L.w8a8_attn_decode(FAKE, 3, 0, 1, FAKE, FAKE, FAKE, FAKE, 8, FAKE, None, 0, None) == w8a8.EUNSUPPORTED
        assert L.w8a8_attn_decode(FAKE, 4, 9, 1, FAKE, FAKE, FAKE, FAKE, 8, FAKE, None, 0, None) == w8a8.EINVAL
        assert L.w8a8_ffn_stack_status(None, 1 << 20, None) == w8a8.EINVAL
        for s in range(-1, 8):
            L.w8a8_status_str(s)
        buf = (ctypes.c_uint8 * 64)()
        for name in (b"bf16", b"5+5", b"10+10", b"all26", b"nope", b""):
            L.w8a8_precision_map(name, buf, 26)
        db = np.array([30.0, np.nan, 12.0, np.inf, -np.inf, 30.0], np.float32)
        order = np.zeros(6, np.int32)
        assert L.w8a8_rank_layers(db.ctypes.data_as(ctypes.c_void_p), 6,
                                  order.ctypes.data_as(ctypes.c_void_p)) == 0
        assert L.w8a8_set_plan_override(b"NOT_A_KNOB", 1) == -1
        assert L.w8a8_set_plan_override(b"GEMM_SPLITS", 7) == 0
        L.w8a8_linear_workspace_bytes(128, 1152, 6912)
        L.w8a8_clear_plan_overrides()
        print("host ok")
    """ % lib)
    out = _run_child(code, {"LD_PRELOAD": _clang_asan_runtime()})
    assert "host ok" in out
