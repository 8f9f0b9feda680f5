"""Host sanitizer runs (CPU only): the fp64 oracle and the C ABI's argument
validation built with AddressSanitizer and UndefinedBehaviorSanitizer.

* The oracle: every entry point runs once on small inputs under both
  sanitizers (with leak detection), and its outputs are compared bit for bit
  with the same calls through the normal build.
* The ABI: api.cpp (validation, scratch cap, host-only queries) built with
  both sanitizers and linked with the library's kernel objects; a driver
  makes calls that validation rejects, empty calls and capped calls, so no
  kernel is launched and no device is needed."""

import glob
import os
import shutil
import struct
import subprocess

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HERE = os.path.join(ROOT, "tests", "sanitize")
SAN = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer",
       "-g", "-O1"]
ENV = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0",
           UBSAN_OPTIONS="print_stacktrace=1", OMP_NUM_THREADS="2")


def _have(tool):
    return shutil.which(tool) is not None


def _run(cmd, env=None, timeout=300):
    r = subprocess.run(cmd, capture_output=True, text=True, env=env, timeout=timeout)
    assert r.returncode == 0, f"{' '.join(cmd[:3])}... rc={r.returncode}\n{r.stdout}\n{r.stderr}"
    return r


def _read_records(path):
    types = {1: np.uint16, 2: np.uint8, 3: np.float32, 4: np.float64, 5: np.int32}
    out = {}
    with open(path, "rb") as f:
        data = f.read()
    o = 0
    while o < len(data):
        (n,) = struct.unpack_from("<I", data, o)
        o += 4
        name = data[o:o + n].decode()
        o += n
        t, nb = struct.unpack_from("<IQ", data, o)
        o += 12
        out[name] = np.frombuffer(data[o:o + nb], dtype=types[t]).copy()
        o += nb
    return out


@pytest.mark.skipif(not _have("gcc"), reason="gcc not available")
def test_oracle_under_asan_ubsan(tmp_path):
    exe = str(tmp_path / "oracle_san")
    _run(["gcc", "-std=c11", "-fopenmp", *SAN, os.path.join(ROOT, "oracle", "moe_oracle.c"),
          os.path.join(HERE, "oracle_driver.c"), "-o", exe, "-lm"])
    dump = str(tmp_path / "oracle.bin")
    r = _run([exe, dump], env=ENV)
    assert "all entry points ran" in r.stdout
    R = _read_records(dump)

    from oracle import oracle as oracle_mod

    o = oracle_mod.get()
    T, d, ffn, E, k = 13, 128, 192, 8, 2
    x = R["x"].reshape(T, d)
    wr = R["wr"].reshape(E, d)
    w1, w3 = R["w1"].reshape(E, ffn, d), R["w3"].reshape(E, ffn, d)
    w2 = R["w2"].reshape(E, d, ffn)
    logits = o.router_logits(x, wr, R["bias"])
    assert np.array_equal(logits.reshape(-1), R["logits"])
    ids, gates = o.topk_gate(logits, k)
    assert np.array_equal(ids.reshape(-1), R["ids"]) and np.array_equal(gates.reshape(-1), R["gates"])
    g2 = o.gates_for_ids(logits, R["ids2"].reshape(T, k))
    assert np.array_equal(g2.reshape(-1), R["gates2"])
    counts, offs, perm = o.dispatch(ids, E)
    assert np.array_equal(counts, R["counts"]) and np.array_equal(offs, R["offsets"])
    assert np.array_equal(perm, R["perm"])
    out, h, y = o.moe_apply(x, w1, w3, w2, ids, gates, want_slots=True)
    assert np.array_equal(out.reshape(-1), R["apply_out"])
    assert np.array_equal(h.reshape(-1), R["apply_h"]) and np.array_equal(y.reshape(-1), R["apply_y"])
    lay = o.moe_layer(x, wr, w1, w3, w2, k, R["bias"])
    assert np.array_equal(lay["out"].reshape(-1), R["layer_out"])
    q1, q3 = R["q1"].reshape(E, ffn, d), R["q3"].reshape(E, ffn, d)
    q2 = R["q2"].reshape(E, d, ffn)
    s1, s3, s2 = R["s1"].reshape(E, ffn), R["s3"].reshape(E, ffn), R["s2"].reshape(E, d)
    assert np.array_equal(o.fp8_e4m3(np.arange(256, dtype=np.uint8)), R["e4m3_all"], equal_nan=True)
    out8, h8, _ = o.moe_apply_fp8(x, q1, s1, q3, s3, q2, s2, ids, gates, want_slots=True)
    assert np.array_equal(out8.reshape(-1), R["apply8_out"])
    assert np.array_equal(h8.reshape(-1), R["apply8_h"])
    lay8 = o.moe_layer_fp8(x, wr, q1, s1, q3, s3, q2, s2, k)
    assert np.array_equal(lay8["out"].reshape(-1), R["layer8_out"])
    a = o.rmsnorm(R["hres"].reshape(T, d), R["gamma"], 1e-5)
    assert np.array_equal(a.reshape(-1), R["rms"])
    assert np.array_equal(o.round_bf16(a).reshape(-1), R["rms_bf16"])
    q = R["q_in"].reshape(3, 4, 16).copy()
    qr = o.rope(q, R["pos"], 10000.0)
    assert np.array_equal(qr.reshape(-1), R["q_rope"])
    kc, vc = R["kc"].reshape(10, 2, 8, 16), R["vc"].reshape(10, 2, 8, 16)
    att = o.attention_decode(qr, kc, vc, R["pt"].reshape(3, 4), R["ctx"], 0.25)
    assert np.array_equal(att.reshape(-1), R["attn"])


@pytest.mark.skipif(not (_have("g++") and os.path.exists("/opt/rocm/include/hip/hip_runtime.h")),
                    reason="g++ or the HIP headers are not available")
def test_abi_validation_under_asan_ubsan(tmp_path):
    from paper_2408_00008_amd import build

    objs = [o for o in glob.glob(os.path.join(build.BUILD, "*.hip.o"))]
    if len(objs) < len(glob.glob(os.path.join(build.CSRC, "*.hip"))):
        build.build()
        objs = glob.glob(os.path.join(build.BUILD, "*.hip.o"))
    inc = ["-D__HIP_PLATFORM_AMD__", "-I/opt/rocm/include", "-I" + os.path.join(ROOT, "include"),
           "-I" + build.CSRC]
    api_o = str(tmp_path / "api_san.o")
    _run(["g++", "-std=c++17", *SAN, *inc, "-c", os.path.join(build.CSRC, "api.cpp"), "-o", api_o])
    exe = str(tmp_path / "abi_san")
    _run(["g++", "-std=c++17", *SAN, *inc, os.path.join(HERE, "abi_driver.cpp"), api_o, *objs,
          "-o", exe, "-L/opt/rocm/lib", "-Wl,-rpath,/opt/rocm/lib", "-lamdhip64"])
    # the HIP runtime's own allocations at exit are not this library's leaks
    supp = tmp_path / "lsan.supp"
    supp.write_text("leak:libamdhip64\nleak:libhsa-runtime64\nleak:librocprofiler\n")
    env = dict(ENV, LSAN_OPTIONS=f"suppressions={supp}")
    r = _run([exe], env=env)
    assert "0 failed" in r.stdout, r.stdout + r.stderr
