"""Convs whose weight fragments go through the LDS ring (wconv_kernel) against
the same decoder with every weight fragment loaded per wave (DC_NO_RING).

Both paths use one K partition and the same channel block for each conv and
add each output's MFMA products in the same (channel block, tap, chunk)
order, so the PCM must agree bit for bit -- with fused resblock pairs and
without, for chunked calls that carry state and for a call of another size.
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


@pytest.mark.parametrize("batch,flags", [(8, dc.DC_NO_FUSE), (16, dc.DC_NO_FUSE), (64, 0)])
def test_ring_equals_register_weights(batch, flags):
    arch = synth.REAL_ARCH
    blob = synth.make_weights(arch, 0)
    n = 25
    sizes = [n, n, 9, n]
    ids = synth.make_tokens(arch, batch, sum(sizes))
    say(f"ring vs register weights, real bf16, batch {batch}, flags {flags}, calls {sizes}")
    ring = dc.Decoder(arch, "bf16", blob, batch=batch, chunk_tokens=n, flags=flags)
    plain = dc.Decoder(arch, "bf16", blob, batch=batch, chunk_tokens=n, flags=flags | dc.DC_NO_RING)
    kr = [l["kernel"] for l in ring.layers()]
    kp = [l["kernel"] for l in plain.layers()]
    say(f"ring kernels: {sum(k.startswith('dc::wconv_kernel') for k in kr)} of {len(kr)} launches")
    assert any(k.startswith("dc::wconv_kernel") for k in kr), kr
    assert not any(k.startswith("dc::wconv_kernel") for k in kp), kp
    a = decode(ring, ids, sizes)
    b = decode(plain, ids, sizes)
    assert np.isfinite(a).all()
    assert bits_equal(a, b), f"ring and register-weight PCM differ (max |d| {np.abs(a - b).max():.3e})"
    ring.close()
    plain.close()
    say(f"batch {batch}: ring == register weights bit for bit ({a.shape[1]} samples per stream)")
