"""Compile libdc.so (the C-ABI library) for gfx950 with hipcc, in-tree."""
from __future__ import annotations

import os
import subprocess
from concurrent.futures import ThreadPoolExecutor

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
LIB = os.path.join(PKG, "libdc.so")
SOURCES = ["dc_runtime.hip", "dc_kernels.hip", "flow_runtime.hip", "flow_kernels.hip"]

HIPCC_FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC",
    # packed fp32 VALU forms stay off: ordinary float code only
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wno-unused-command-line-argument",
]

# the host pass does not know the (device) feature flag: drop that notice
_NOISE = "'-packed-fp32-ops' is not a recognized feature"


def _run(cmd, verbose):
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    msg = "\n".join(l for l in (r.stdout + r.stderr).splitlines() if _NOISE not in l)
    if msg.strip():
        print(msg, flush=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed ({r.returncode}): {cmd[-1]}")


DEBUG_LIB = os.path.join(PKG, "libdc_debug.so")


def build(verbose: bool = False, out: str = LIB, defines=(), debug: bool = True) -> str:
    """Compile every source to an object in parallel (they share no device
    code), then link the shared library; with `debug`, also the checked
    library libdc_debug.so: the vocoder kernels built with DC_DEBUG (bounds
    checks on every ring access) linked with the same other objects."""
    hipcc = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
    objdir = os.path.join(PKG, "_build")
    os.makedirs(objdir, exist_ok=True)
    tag = os.path.basename(out).replace(".", "_")
    objs = [os.path.join(objdir, f"{tag}_{os.path.splitext(s)[0]}.o") for s in SOURCES]
    inc = ["-I", os.path.join(ROOT, "include")]
    cmds = [[hipcc, *HIPCC_FLAGS, *[f"-D{d}" for d in defines], *inc,
             "-c", "-o", o, os.path.join(CSRC, s)] for s, o in zip(SOURCES, objs)]
    dbg_obj = os.path.join(objdir, "libdc_debug_dc_kernels.o")
    if debug:
        cmds.append([hipcc, *HIPCC_FLAGS, "-DDC_DEBUG", *inc, "-c", "-o", dbg_obj,
                     os.path.join(CSRC, "dc_kernels.hip")])
    with ThreadPoolExecutor(max_workers=len(cmds)) as ex:
        for f in [ex.submit(_run, c, verbose) for c in cmds]:
            f.result()
    links = [(out, objs)]
    if debug:
        links.append((DEBUG_LIB, [dbg_obj if s == "dc_kernels.hip" else o for s, o in zip(SOURCES, objs)]))
    for lib, lobjs in links:
        tmp = lib + ".tmp"
        _run([hipcc, "--offload-arch=gfx950", "-shared", "-fPIC", "-o", tmp, *lobjs], verbose)
        os.replace(tmp, lib)
    return out


if __name__ == "__main__":
    print(build(verbose=True))
