"""The host code of both runtimes under AddressSanitizer and
UndefinedBehaviorSanitizer: dc_runtime.hip and flow_runtime.hip are compiled
with the sanitizers on their host side only (the kernels are the library's
own objects, unsanitized), linked with tests/asan_driver.cpp, and the driver
walks dc_init / dc_flow_init over several hundred valid and invalid
configurations and every entry point's NULL-state path.  Without a GPU a
valid configuration runs the whole host set-up (validation, network, tile
choice, schedule, arena layout) up to the first device allocation."""
from __future__ import annotations

import os
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2609_35115_amd", "csrc")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
CLANG = "/opt/rocm/llvm/bin/clang++"
# host-side sanitizers only: each -fsanitize= behind -Xarch_host
SAN_HOST = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
            "-Xarch_host", "-fno-sanitize-recover=all"]


def _run(cmd, **kw):
    r = subprocess.run(cmd, capture_output=True, text=True, **kw)
    msg = "\n".join(l for l in (r.stdout + r.stderr).splitlines() if "packed-fp32-ops" not in l)
    assert r.returncode == 0, f"{' '.join(cmd[:3])} ...: {msg[-4000:]}"
    return r


def test_runtimes_under_address_and_undefined_behaviour_sanitizers(tmp_path):
    if not (os.path.exists(HIPCC) and os.path.exists(CLANG)):
        pytest.skip("hipcc or ROCm's clang++ is not installed")
    from paper_2609_35115_amd import _build
    objdir = os.path.join(ROOT, "paper_2609_35115_amd", "_build")
    kernels = [os.path.join(objdir, f"libdc_so_{n}.o") for n in ("dc_kernels", "flow_kernels")]
    if not all(os.path.exists(k) for k in kernels):
        _build.build()
    objs = []
    for src in ("dc_runtime.hip", "flow_runtime.hip"):
        o = str(tmp_path / (os.path.splitext(src)[0] + ".o"))
        _run([HIPCC, "--offload-arch=gfx950", "-O1", "-g", "-std=c++17", "-fPIC",
              "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops", *SAN_HOST,
              "-I", os.path.join(ROOT, "include"), "-c", os.path.join(CSRC, src), "-o", o])
        objs.append(o)
    drv = str(tmp_path / "driver.o")
    _run([CLANG, "-O1", "-g", "-std=c++17", "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
          "-I", os.path.join(ROOT, "include"), "-c", os.path.join(ROOT, "tests", "asan_driver.cpp"), "-o", drv])
    exe = str(tmp_path / "driver")
    _run([CLANG, "-fsanitize=address,undefined", "-o", exe, drv, *objs, *kernels,
          "-L/opt/rocm/lib", "-lamdhip64", "-Wl,-rpath,/opt/rocm/lib"])
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=0:abort_on_error=1",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    r = subprocess.run([exe], env=env, capture_output=True, text=True, timeout=600)
    report = r.stdout + r.stderr
    assert r.returncode == 0, report[-4000:]
    assert "failures 0" in r.stdout, report[-4000:]
    assert "runtime error" not in report and "AddressSanitizer" not in report, report[-4000:]
