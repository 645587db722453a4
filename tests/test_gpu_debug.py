"""The checked build (libdc_debug.so: the kernels built with DC_DEBUG, every
ring access and operand-tile row range bounds-checked) against the release
build, on the GPU: across the kernel families -- K-split and batched convs,
the LDS-ring conv, the fused pairs, the harmonic source, the iSTFT tail,
graph replays and direct calls of other sizes, a per-stream reset -- the
checked build must report no failed check and produce the release build's
PCM bit for bit (the checks change no arithmetic)."""
from __future__ import annotations

import os

import numpy as np
import pytest

torch = pytest.importorskip("torch")

import paper_2609_35115_amd as dc  # noqa: E402
from paper_2609_35115_amd import _build, synth  # noqa: E402

from gpu_common import bits_equal, say  # noqa: E402

pytestmark = pytest.mark.gpu

TINY, TINY_NSF, REAL = synth.TINY_ARCH, synth.TINY_NSF_ARCH, synth.REAL_ARCH

# (label, arch, dtype, batch, chunk, max_tokens, call sizes, decoder keywords)
SCENARIOS = [
    ("tiny f32 B=2, replays and direct calls", TINY, "f32", 2, 8, 21, [8, 8, 5, 21], {}),
    ("tiny f32 B=2 with the harmonic source", TINY_NSF, "f32", 2, 8, 8, [8, 8, 3], {}),
    ("real f32 B=1", REAL, "f32", 1, 4, 4, [4, 4, 3], {}),
    ("real bf16 B=1", REAL, "bf16", 1, 2, 3, [2, 2, 3], {}),
    ("real bf16 B=8, fused pairs", REAL, "bf16", 8, 3, 3, [3, 3, 2], {}),
    ("real bf16 B=8, every conv its own launch", REAL, "bf16", 8, 3, 3, [3, 3, 2], {"flags": dc.DC_NO_FUSE}),
    ("real bf16 B=8, LDS-ring conv shape", REAL, "bf16", 8, 3, 3, [3, 2], {"tile_variant": 22}),
]


def _run(label, arch, dtype, batch, chunk, max_tokens, sizes, kw):
    blob = synth.make_weights(arch, 1)
    total = sum(sizes)
    ids = synth.make_tokens(arch, batch, total)
    f0 = synth.make_f0(arch, batch, total) if arch.get("n_harmonics", 0) else None
    fpt = arch["frames_per_token"]
    dec = dc.Decoder(arch, dtype, blob, batch=batch, chunk_tokens=chunk, max_tokens=max_tokens, **kw)
    outs, pos = [], 0
    for i, n in enumerate(sizes):
        if i == len(sizes) - 1 and batch > 1:
            dec.reset_stream(batch - 1)   # a per-stream reset before the last call
        if f0 is not None:
            outs.append(dec.decode(ids[:, pos:pos + n], f0[:, pos * fpt:(pos + n) * fpt]))
        else:
            outs.append(dec.decode(ids[:, pos:pos + n]))
        pos += n
    dec.sync()
    pcm = np.concatenate([o.cpu().numpy() for o in outs], axis=1)
    dec.close()
    return pcm


def test_checked_build_reports_nothing_and_matches_release():
    if not os.path.exists(_build.DEBUG_LIB):
        pytest.fail(f"{_build.DEBUG_LIB} is missing: build it with __graft_entry__.build()")
    assert dc.lib().dc_debug_checks(0) == -1, "the release build must have the checks compiled out"
    release = []
    for sc in SCENARIOS:
        say(f"release: {sc[0]}")
        release.append(_run(*sc))
    saved = (dc._lib, dc.LIB_PATH)
    try:
        dc._lib, dc.LIB_PATH = None, _build.DEBUG_LIB
        assert dc.lib().dc_debug_checks(1) >= 0, "the checked build must report its checks"
        for sc, ref in zip(SCENARIOS, release):
            say(f"checked: {sc[0]}")
            pcm = _run(*sc)
            bits = dc.lib().dc_debug_checks(1)
            assert bits == 0, f"{sc[0]}: failed bounds checks, bits {bits:#x}"
            assert bits_equal(pcm, ref), f"{sc[0]}: checked build differs from release"
    finally:
        dc._lib, dc.LIB_PATH = saved
