"""Fused resblock pairs (the first conv's output kept on chip) against the
same decoder with every conv as its own launch (DC_NO_FUSE).

Both paths run each conv with one K partition and a channel block of all its
channels, so the PCM must agree bit for bit -- on every stream, for chunked
calls that carry state across chunk boundaries, from a fresh state and after
a reset of one stream.
"""
from __future__ import annotations

import numpy as np
import pytest

import paper_2609_35115_amd as dc
from paper_2609_35115_amd import synth
from tests.gpu_common import bits_equal, say

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


def decode(dec, ids, sizes):
    outs, pos = [], 0
    for m in sizes:
        outs.append(dec.decode(ids[:, pos:pos + m]).cpu().numpy())
        pos += m
    dec.sync()
    return np.concatenate(outs, axis=1)


@pytest.mark.parametrize("batch", [8, 16])
def test_fused_pairs_equal_unfused(batch):
    arch = synth.REAL_ARCH
    blob = synth.make_weights(arch, 0)
    n = 25
    sizes = [n, n, 7, n, n]          # replays and one direct call of another size
    ids = synth.make_tokens(arch, batch, sum(sizes))
    say(f"fused vs unfused real bf16, batch {batch}, calls {sizes}")
    fused = dc.Decoder(arch, "bf16", blob, batch=batch, chunk_tokens=n)
    plain = dc.Decoder(arch, "bf16", blob, batch=batch, chunk_tokens=n, flags=dc.DC_NO_FUSE)
    kf = fused.stats()["kernels_per_step"]
    kp = plain.stats()["kernels_per_step"]
    say(f"launches per step: fused {kf}, unfused {kp}")
    assert kf < kp
    names = [l["kernel"] for l in fused.layers()]
    assert any(k.startswith("dc::pair_kernel") for k in names), names
    a = decode(fused, ids, sizes)
    b = decode(plain, ids, sizes)
    assert bits_equal(a, b), "fused and unfused PCM differ"
    # one stream reset, then more chunks: still identical
    fused.reset_stream(batch // 2)
    plain.reset_stream(batch // 2)
    more = synth.make_tokens(arch, batch, 2 * n)[:, ::-1].copy()
    a2 = decode(fused, more, [n, n])
    b2 = decode(plain, more, [n, n])
    assert bits_equal(a2, b2), "fused and unfused PCM differ after reset_stream"
    # the fused pair's h holds no frames; the z ring beside it does
    last = (sum(sizes) + 2 * n) * synth.samples_per_token(arch) // 4 - 1
    z = fused.tap("s2.rb0.z0", 0, last, 1)
    assert z.shape == (1, 64) and np.isfinite(z).all()
    with pytest.raises(dc.DcError) as ei:
        fused.tap("s2.rb0.h0", 0, last, 1)
    assert ei.value.status == dc.DC_ERANGE
    fused.close()
    plain.close()
    say(f"batch {batch}: fused == unfused bit for bit ({a.shape[1] + a2.shape[1]} samples per stream)")
