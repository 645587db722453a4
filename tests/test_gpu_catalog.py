"""Partial-chunk shape classes (DC_FLUSH_CATALOG): every n below the chunk size
replays its own captured graph, and the PCM is bit-identical to direct
launches and to the offline decode, and within tolerance of the oracle --
also for a stream reset in place between replays."""
from __future__ import annotations

import numpy as np
import pytest

import oracle
import paper_2609_35115_amd as dc
from paper_2609_35115_amd import synth
from tests.gpu_common import TOL, bits_equal, err_stats, say

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


def run(dec, ids, sizes):
    outs, pos = [], 0
    for n in sizes:
        outs.append(dec.decode(ids[:, pos:pos + n]))
        pos += n
    dec.sync()
    return np.concatenate([o.cpu().numpy() for o in outs], axis=1)


@pytest.mark.parametrize("arch_name,dtype,batch,chunk,sizes", [
    ("tiny", "f32", 2, 8, [8, 3, 8, 1, 7, 8, 5]),
    ("real", "bf16", 8, 6, [6, 2, 6, 5, 1, 6]),
])
def test_flush_classes_replay_bit_exact(arch_name, dtype, batch, chunk, sizes):
    arch = synth.TINY_ARCH if arch_name == "tiny" else synth.REAL_ARCH
    blob = synth.make_weights(arch, 0)
    total = sum(sizes)
    ids = synth.make_tokens(arch, batch, total)
    say(f"{arch_name} {dtype} B={batch} chunk {chunk}: calls {sizes}")
    cat = dc.Decoder(arch, dtype, blob, batch=batch, chunk_tokens=chunk, max_tokens=chunk + 2,
                     flags=dc.DC_FLUSH_CATALOG)
    st = cat.stats()
    assert st["graph_classes"] == chunk
    got = run(cat, ids, sizes)
    st = cat.stats()
    flushes = sum(1 for n in sizes if n < chunk)
    assert st["replays"] == len(sizes) and st["replays_flush"] == flushes and st["direct_shape"] == 0

    plain = dc.Decoder(arch, dtype, blob, batch=batch, chunk_tokens=chunk)
    assert plain.stats()["graph_classes"] == 1
    ref = run(plain, ids, sizes)
    assert plain.stats()["direct_shape"] == flushes
    assert bits_equal(got, ref), "catalog replay differs from direct launches"

    # offline: the whole sequence in one call of a state with the same chunk
    # size (the arithmetic is fixed by the layer shapes, batch and chunk size)
    off = dc.Decoder(arch, dtype, blob, batch=batch, chunk_tokens=chunk, max_tokens=total)
    whole = run(off, ids, [total])
    assert bits_equal(got, whole), "catalog replay differs from the offline decode"

    # a call above the chunk size is still admitted and runs directly
    cat.reset()
    more = synth.make_tokens(arch, batch, chunk + 2)
    cat.decode(more)
    cat.sync()
    assert cat.stats()["direct_shape"] == 1
    for d in (cat, plain, off):
        d.close()


@pytest.mark.parametrize("arch_name,dtype,batch,chunk,sizes", [
    ("tiny", "f32", 2, 8, [8, 3, 8, 1, 7, 8, 5]),
    ("real", "bf16", 8, 6, [6, 2, 6, 5, 1, 6]),
])
def test_flush_classes_match_the_oracle(arch_name, dtype, batch, chunk, sizes):
    """The replayed partial-chunk classes (Eq. catalog, Eq. width: one class per
    admissible n below the chunk) against the fp64 oracle's offline decode of
    each stream, within the workload tolerance."""
    arch = synth.TINY_ARCH if arch_name == "tiny" else synth.REAL_ARCH
    blob = synth.make_weights(arch, 0)
    total = sum(sizes)
    ids = synth.make_tokens(arch, batch, total, seed=3)
    cat = dc.Decoder(arch, dtype, blob, batch=batch, chunk_tokens=chunk, max_tokens=chunk + 2,
                     flags=dc.DC_FLUSH_CATALOG)
    got = run(cat, ids, sizes)
    assert cat.stats()["replays_flush"] == sum(1 for n in sizes if n < chunk)
    cat.close()
    worst = 0.0
    for b in range(batch):
        ref = oracle.decode(arch, dtype, blob, ids[b])
        e, _ = err_stats(got[b], ref)
        worst = max(worst, e)
        assert e <= TOL[dtype], f"stream {b}: {e:.3e}"
    say(f"{arch_name} {dtype} catalog replays vs oracle: worst max-abs/RMS {worst:.3e}")


@pytest.mark.parametrize("arch_name,dtype,batch,chunk", [("tiny", "f32", 3, 8), ("real", "bf16", 8, 6)])
def test_stream_reset_under_replay_matches_a_fresh_oracle_stream(arch_name, dtype, batch, chunk):
    """dc_reset_stream in the middle of replayed calls (full and partial
    classes): the reset stream continues as a fresh stream of the oracle, the
    others as their uninterrupted oracle streams."""
    arch = synth.TINY_ARCH if arch_name == "tiny" else synth.REAL_ARCH
    blob = synth.make_weights(arch, 1)
    before, after = [chunk, 3], [chunk, 2, chunk]
    nb, na = sum(before), sum(after)
    ids = synth.make_tokens(arch, batch, nb + na, seed=4)
    dec = dc.Decoder(arch, dtype, blob, batch=batch, chunk_tokens=chunk, max_tokens=chunk,
                     flags=dc.DC_FLUSH_CATALOG)
    run(dec, ids[:, :nb], before)
    r = batch - 1
    dec.reset_stream(r)
    got = run(dec, ids[:, nb:], after)
    st = dec.stats()
    assert st["replays"] == len(before) + len(after) and st["direct_shape"] == 0, st
    dec.close()
    spt = synth.samples_per_token(arch)
    for b in (0, r):
        if b == r:
            ref = oracle.decode(arch, dtype, blob, ids[b, nb:])
        else:
            ref = oracle.decode(arch, dtype, blob, ids[b])[nb * spt:]
        e, _ = err_stats(got[b], ref)
        say(f"{arch_name} {dtype} stream {b} ({'reset' if b == r else 'continued'}): max-abs/RMS {e:.3e}")
        assert e <= TOL[dtype], f"stream {b}: {e:.3e}"
