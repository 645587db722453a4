"""The oracle's C code under AddressSanitizer and UndefinedBehaviorSanitizer
(host code, gcc): a child process with the sanitizer runtime preloaded drives
the sanitized library through the oracle's own Python API -- the vocoder
decode (tiny architecture, with and without the harmonic source, with taps),
its library-checkable pieces (causal and transposed conv, inverse real DFT,
iSTFT) and a tiny flow-decoder turn (prompt, lookahead calls, a flush, the
carry) -- and any out-of-bounds access, use after free or undefined
operation ends it with a report."""
from __future__ import annotations

import os
import subprocess
import sys
import textwrap

import pytest

import oracle

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

DRIVER = textwrap.dedent("""
    import numpy as np
    import oracle
    from paper_2609_35115_amd import synth

    rng = np.random.default_rng(0)
    W, b, v = rng.standard_normal((5, 4, 3)), rng.standard_normal(5), rng.standard_normal((4, 9))
    oracle.cconv(W, b, v, 2)
    oracle.convt(rng.standard_normal((4, 5, 6)), b, v)
    oracle.irfft(rng.standard_normal(9), rng.standard_normal(9))
    oracle.istft(rng.standard_normal((7, 9)), rng.standard_normal((7, 9)))   # [frames][bins]
    for arch in (synth.TINY_ARCH, synth.TINY_NSF_ARCH):
        blob = synth.make_weights(arch, 0)
        ids = synth.make_tokens(arch, 1, 12)[0]
        kw = {}
        if arch.get("n_harmonics", 0):
            kw = dict(f0=synth.make_f0(arch, 1, 12)[0], seed=3, stream=1)
        for dtype in ("f32", "bf16"):
            oracle.decode(arch, dtype, blob, ids, **kw)
        oracle.decode(arch, "f32", blob, ids, tap="s1.rb0.h1", **kw)
        oracle.decode(arch, "f32", blob, ids, tap="head", **kw)
    a = synth.TINY_FLOW_ARCH
    s = oracle.FlowStream(a, "bf16", synth.make_flow_weights(a, 0), seed=2, key=1)
    s.prompt(*synth.make_flow_prompt(a, a["f_prompt"]))
    mu = synth.make_flow_mu(a, 1, 5 * a["f_chunk"] + a["f_call"])[0]
    for k in range(4):
        s.chunk(mu[k * a["f_chunk"]:k * a["f_chunk"] + a["f_call"]])
    s.chunk(mu[:3])
    s.carry(1, 1, 0, 1)
    print("sanitized oracle run ok", flush=True)
""")


def test_oracle_under_address_and_undefined_behaviour_sanitizers(tmp_path):
    asan = subprocess.run(["gcc", "-print-file-name=libasan.so"], capture_output=True, text=True).stdout.strip()
    if not os.path.isabs(asan) or not os.path.exists(asan):
        pytest.skip("gcc's AddressSanitizer runtime is not installed")
    lib = oracle.build_sanitized(str(tmp_path / "liboracle_san.so"))
    env = dict(os.environ, DC_ORACLE_LIB=lib, LD_PRELOAD=asan, PYTHONPATH=ROOT,
               ASAN_OPTIONS="detect_leaks=0:abort_on_error=1", UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    r = subprocess.run([sys.executable, "-c", DRIVER], env=env, capture_output=True, text=True, timeout=600)
    report = r.stdout + r.stderr
    assert r.returncode == 0, report[-4000:]
    assert "sanitized oracle run ok" in r.stdout
    assert "runtime error" not in report and "AddressSanitizer" not in report, report[-4000:]
