"""The library's host code under AddressSanitizer and UndefinedBehaviorSanitizer (CPU only).

tests/asan/driver.cpp is built against the library sources with the sanitizers on
the host pass (device code is compiled as usual and never run).  It reads model
descriptors dumped here -- the seven workloads, hand-made invalid descriptors and
random corruptions of valid ones -- and drives every host-only entry point: model
creation and validation, both layer profiles, planning over them, workspace and
code sizes, cut tensors, timing slots; then the planner and the sub-slice ranges on
random inputs.  Any sanitizer report or failed check fails the test.
"""
import ctypes
import os
import shutil
import struct
import subprocess
from concurrent.futures import ThreadPoolExecutor

import numpy as np
import pytest

import synth
from tests.helpers import SMALL

P = pytest.importorskip("paper_2404_02445_amd")
from paper_2404_02445_amd import _lib as L  # noqa: E402
from paper_2404_02445_amd import binding as B  # noqa: E402

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2404_02445_amd", "csrc")
BUILD = os.path.join(ROOT, "tests", "asan", "_build")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
SOURCES = [os.path.join(CSRC, f) for f in ("abi.cpp", "plan.cpp", "model.cpp", "gemm.hip", "kernels.hip",
                                           "lstm.hip", "noalloc.hip")] + [os.path.join(ROOT, "tests", "asan", "driver.cpp")]
# sanitizers on the host pass only (each flag directly after -Xarch_host)
HOST_SAN = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
            "-Xarch_host", "-fno-sanitize-recover=undefined", "-Xarch_host", "-fno-omit-frame-pointer"]
FLAGS = ["-x", "hip", "--offload-arch=gfx950", "-std=c++17", "-O1", "-g",
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]


def _obj(src):
    return os.path.join(BUILD, os.path.basename(src) + ".o")


def _compile(src):
    obj = _obj(src)
    deps = [src, os.path.join(CSRC, "internal.h"), os.path.join(ROOT, "include", "mopar.h")]
    if os.path.exists(obj) and os.path.getmtime(obj) >= max(os.path.getmtime(d) for d in deps):
        return obj
    r = subprocess.run([HIPCC, *FLAGS, *HOST_SAN, "-c", src, "-o", obj], capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{r.stderr[-3000:]}")
    return obj


@pytest.fixture(scope="module")
def driver():
    if not shutil.which(HIPCC):
        pytest.skip("hipcc not found")
    os.makedirs(BUILD, exist_ok=True)
    with ThreadPoolExecutor(max_workers=4) as ex:
        objs = list(ex.map(_compile, SOURCES))
    exe = os.path.join(BUILD, "driver")
    if not os.path.exists(exe) or os.path.getmtime(exe) < max(os.path.getmtime(o) for o in objs):
        r = subprocess.run([HIPCC, "--offload-arch=gfx950", *HOST_SAN, *objs, "-o", exe], capture_output=True, text=True)
        if r.returncode != 0:
            raise RuntimeError("link failed:\n" + r.stderr[-3000:])
    return exe


def _dump(path, tens, ops, d, weights_bytes, expect_ok):
    """The descriptor as the driver reads it: header, then the raw C structs."""
    size_check = ctypes.sizeof(L.TensorDesc) * 1000 + ctypes.sizeof(L.Op)
    with open(path, "wb") as f:
        f.write(b"MOPD")
        f.write(struct.pack("<8i", 1, expect_ok, d["dtype"], len(tens), len(ops), d["n_layers"], d["input"],
                            size_check))
        f.write(struct.pack("<iq", d["output"], weights_bytes))
        f.write(bytes(tens))
        f.write(bytes(ops))


def _packed(m):
    tens, ops, blob = B._pack(m)
    d = dict(dtype=B.DTYPE[m.dtype], n_layers=len(m.layers), input=m.input_tid, output=m.output_tid)
    return tens, ops, d, blob.size


def _copy(arr):
    out = (arr._type_ * len(arr))()
    ctypes.memmove(out, arr, ctypes.sizeof(arr))
    return out


def _invalid_variants(m):
    """Hand-made invalid descriptors of model m: (name, tensors, ops, header, weights_bytes)."""
    tens, ops, d, wb = _packed(m)
    n_t = len(tens)
    later = next(i for i in range(len(ops)) if ops[i].layer >= 1)
    conv = next(i for i in range(len(ops)) if ops[i].kind == L.OP_CONV)

    def mut(name, f, **hdr):
        t2, o2 = _copy(tens), _copy(ops)
        f(t2, o2)
        return name, t2, o2, dict(d, **hdr), wb

    return [
        mut("tensor id out of range", lambda t, o: setattr(o[1], "in0", n_t + 5)),
        mut("negative tensor id", lambda t, o: setattr(o[1], "out", -3)),
        mut("decreasing layer", lambda t, o: setattr(o[later + 1], "layer", 0) if later + 1 < len(o) else None),
        mut("weight offset past the blob", lambda t, o: setattr(o[conv], "w", wb + 64)),
        mut("misaligned weight offset", lambda t, o: setattr(o[conv], "w", 3)),
        mut("zero dimension", lambda t, o: t[2].dims.__setitem__(1, 0)),
        mut("rank 5", lambda t, o: setattr(t[2], "rank", 5)),
        mut("zero kernel size", lambda t, o: setattr(o[conv], "kh", 0)),
        mut("zero outputs", lambda t, o: setattr(o[conv], "n_out", 0)),
        mut("unknown op kind", lambda t, o: setattr(o[1], "kind", 99)),
        mut("unknown activation", lambda t, o: setattr(o[conv], "act", 7)),
        mut("output is the input", lambda t, o: None, output=d["input"]),
        mut("a node without ops", lambda t, o: None, n_layers=d["n_layers"] + 1),
        mut("output not from the last op", lambda t, o: setattr(o[len(o) - 1], "out", o[len(o) - 2].out)),
        mut("bad model dtype", lambda t, o: None, dtype=7),
    ]


def test_host_code_under_sanitizers(driver, tmp_path):
    paths = []
    models = [synth.build(c, **SMALL[c]) for c in range(1, 8)] + [synth.build(1), synth.build(2), synth.build(4),
                                                                   synth.build(5)]
    for i, m in enumerate(models):
        tens, ops, d, wb = _packed(m)
        p = tmp_path / f"ok{i}.bin"
        _dump(p, tens, ops, d, wb, 1)
        paths.append(str(p))
    for j, (name, tens, ops, d, wb) in enumerate(_invalid_variants(models[1])):
        p = tmp_path / f"bad{j}.bin"
        _dump(p, tens, ops, d, wb, 0)
        paths.append(str(p))
    # random corruptions of one int32 field of one op: accepted or refused, never a crash
    rng = np.random.default_rng(7)
    for j in range(300):
        m = models[int(rng.integers(0, 7))]
        tens, ops, d, wb = _packed(m)
        o2 = _copy(ops)
        raw = (ctypes.c_int32 * (ctypes.sizeof(o2) // 4)).from_buffer(o2)
        op = int(rng.integers(0, len(o2)))
        word = op * (ctypes.sizeof(L.Op) // 4) + int(rng.integers(0, 19))   # the int32 fields before eps
        raw[word] = int(rng.choice([-1, 0, 1, 2, 3, 7, 64, 1 << 20, -(1 << 30), int(rng.integers(-50, 50))]))
        p = tmp_path / f"fuzz{j}.bin"
        _dump(p, tens, o2, d, wb, 2)
        paths.append(str(p))
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0", UBSAN_OPTIONS="print_stacktrace=1")
    r = subprocess.run([driver, *paths], capture_output=True, text=True, env=env, timeout=600)
    out = r.stdout + r.stderr
    assert "AddressSanitizer" not in out and "runtime error" not in out and "LeakSanitizer" not in out, out[-4000:]
    assert r.returncode == 0, out[-4000:]
    assert f"{len(paths)} models, 0 failed checks" in r.stdout
