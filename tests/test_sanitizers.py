"""AddressSanitizer + UBSan builds of the host code, run on the CPU.

The library's host runtime (descriptor validation, shape, byte and workspace
calculus, profiles without timing, split choice, every error path) is built
host-only with the kernel launchers replaced by stubs, and driven over every
model the library ships; the oracle's C library is driven over small
geometries.  Every buffer an entry point writes is a heap block of exactly
its size, so a write past it is reported.  Leak checking is off: the HIP
runtime the library links keeps allocations until exit.
"""
import os
import shutil
import subprocess

import pytest

from paper_2210_08650_amd import binding as B
from paper_2210_08650_amd import models as PM

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SAN = os.path.join(ROOT, "tests", "sanitize")
CSRC = os.path.join(ROOT, "paper_2210_08650_amd", "csrc")
ENV = dict(os.environ, ASAN_OPTIONS="detect_leaks=0:halt_on_error=1",
           UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1", OMP_NUM_THREADS="2")
FIELDS = ("kind", "cin", "cout", "width", "k", "stride", "pad", "relu", "has_bias", "has_bn", "heads", "mlp_dim")


def _hipcc():
    for c in ("/opt/rocm/bin/hipcc", shutil.which("hipcc") or ""):
        if c and os.path.exists(c):
            return c
    pytest.skip("hipcc not found")


def _run(cmd, **kw):
    r = subprocess.run(cmd, capture_output=True, text=True, **kw)
    assert r.returncode == 0, f"{' '.join(cmd[:3])} ...: rc {r.returncode}\n{r.stdout[-3000:]}\n{r.stderr[-3000:]}"
    return r


def test_host_runtime_under_asan_ubsan(tmp_path):
    hipcc = _hipcc()
    # -Xarch_host applies each sanitizer to the host compilation only (the
    # runtime's one device object, the no-allocation scratch array, is built
    # as usual).
    flags = ["-x", "hip", "--offload-arch=gfx950", "-O1", "-g", "-std=c++17", "-I", os.path.join(ROOT, "include"),
             "-I", CSRC, "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
             "-Xarch_host", "-fno-omit-frame-pointer", "-Wno-unused-result"]
    objs = []
    for src in (os.path.join(CSRC, "api.cpp"), os.path.join(CSRC, "split.cpp"), os.path.join(SAN, "stubs.cpp"),
                os.path.join(SAN, "host_driver.cpp")):
        o = str(tmp_path / (os.path.basename(src) + ".o"))
        _run([hipcc] + flags + ["-c", src, "-o", o])
        objs.append(o)
    exe = str(tmp_path / "host_driver")
    _run([hipcc, "--offload-arch=gfx950", "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined"]
         + objs + ["-o", exe])
    spec = tmp_path / "models.txt"
    lines = []
    for name in ("alexnet", "resnet18", "resnet50", "vgg16", "vit_b16", "densenet_block", "densenet121"):
        layers = PM.FACTORIES[name]()
        dt = B.HAPI_F32 if name == "alexnet" else B.HAPI_BF16
        lines.append(f"model {dt} 3 224 224 {len(layers)}")
        for L in layers:
            lines.append(" ".join(str(int(L.get(f, 0))) for f in FIELDS))
    spec.write_text("\n".join(lines) + "\n")
    r = _run([exe, str(spec)], env=ENV, timeout=600)
    assert r.stdout.startswith("OK 7 models"), r.stdout
    assert "runtime error" not in r.stderr and "AddressSanitizer" not in r.stderr, r.stderr[-3000:]


def test_oracle_under_asan_ubsan(tmp_path):
    gcc = shutil.which("gcc")
    if not gcc:
        pytest.skip("gcc not found")
    exe = str(tmp_path / "oracle_driver")
    _run([gcc, "-O1", "-g", "-fopenmp", "-std=c11", "-fsanitize=address,undefined", "-fno-omit-frame-pointer",
          os.path.join(ROOT, "oracle", "oracle.c"), os.path.join(SAN, "oracle_driver.c"), "-o", exe, "-lm"])
    r = _run([exe], env=ENV, timeout=600)
    assert r.stdout.startswith("OK"), r.stdout
    assert "runtime error" not in r.stderr and "AddressSanitizer" not in r.stderr, r.stderr[-3000:]
