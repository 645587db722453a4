"""Carry snapshots (dc_carry_export / dc_carry_import) on the GPU.

A stream's carry is O(1) in its length (Design, state rule, Eq. carry), so a
session can leave a stream slot and continue in another slot, of the same or
another state with the same layout, or rewind to a checkpoint.  Everything a
stream's next call reads from its past travels in the snapshot, so the
continued PCM equals the uninterrupted decode bit for bit -- including the
harmonic source, whose generator key moves with the session -- and the
oracle's decode of the session's own tokens.  One state serves more sessions
than it has slots by time-multiplexing them through snapshots.
"""
from __future__ import annotations

import numpy as np
import pytest

import oracle
import paper_2609_35115_amd as dc
from paper_2609_35115_amd import synth
from tests.gpu_common import TOL, bits_equal, err_stats, say

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


def run(dec, ids, sizes, f0=None):
    fpt = dec.arch["frames_per_token"]
    outs, pos = [], 0
    for n in sizes:
        if f0 is None:
            outs.append(dec.decode(ids[:, pos:pos + n]))
        else:
            outs.append(dec.decode(ids[:, pos:pos + n], f0[:, pos * fpt:(pos + n) * fpt]))
        pos += n
    dec.sync()
    return np.concatenate([o.cpu().numpy() for o in outs], axis=1)


CASES = [
    ("tiny", synth.TINY_ARCH, "f32", 3, 8),
    ("tiny+src", synth.TINY_NSF_ARCH, "f32", 3, 8),
    ("real-bf16-fused", synth.REAL_ARCH, "bf16", 8, 25),
]


@pytest.mark.parametrize("label,arch,dtype,B,n", CASES, ids=[c[0] for c in CASES])
def test_stream_moves_to_another_state_and_slot(label, arch, dtype, B, n):
    blob = synth.make_weights(arch, 1)
    src = arch.get("n_harmonics", 0) > 0
    ids = synth.make_tokens(arch, B, 4 * n, seed=5)
    f0 = synth.make_f0(arch, B, 4 * n, seed=5) if src else None
    other = synth.make_tokens(arch, B, 4 * n, seed=6)
    other_f0 = synth.make_f0(arch, B, 4 * n, seed=6) if src else None
    a = dc.Decoder(arch, dtype, blob, batch=B, chunk_tokens=n, rng_seed=3)
    b = dc.Decoder(arch, dtype, blob, batch=B, chunk_tokens=n, rng_seed=3)
    # a: two chunks, then stream 1 leaves; b: one chunk of other tokens (another clock)
    run(a, ids[:, :2 * n], [n, n], f0[:, :2 * n * arch["frames_per_token"]] if src else None)
    run(b, other[:, :n], [n], other_f0[:, :n * arch["frames_per_token"]] if src else None)
    snap = a.export_carry(1)
    assert snap.size == dc.dc_carry_bytes(a.h)
    b.import_carry(B - 1, snap)
    # both continue with stream 1's next two chunks (in slot B-1 of b)
    fpt = arch["frames_per_token"]
    cont_ids = ids[:, 2 * n:]
    cont_f0 = f0[:, 2 * n * fpt:] if src else None
    pa = run(a, cont_ids, [n, n], cont_f0)
    ids_b = other[:, n:3 * n].copy()
    ids_b[B - 1] = cont_ids[1]
    f0_b = None
    if src:
        f0_b = other_f0[:, n * fpt:3 * n * fpt].copy()
        f0_b[B - 1] = cont_f0[1]
    pb = run(b, ids_b, [n, n], f0_b)
    assert bits_equal(pb[B - 1], pa[1]), f"{label}: moved stream differs from the uninterrupted one"
    # the other streams of b are untouched by the import
    c = dc.Decoder(arch, dtype, blob, batch=B, chunk_tokens=n, rng_seed=3)
    run(c, other[:, :n], [n], other_f0[:, :n * fpt] if src else None)
    pc = run(c, ids_b, [n, n], f0_b)
    assert bits_equal(pb[0], pc[0])
    say(f"{label}: stream moved between states and slots, bit-exact over {pa.shape[1]} samples")
    for d in (a, b, c):
        d.close()


def test_checkpoint_and_rewind():
    arch = synth.REAL_ARCH
    blob = synth.make_weights(arch, 2)
    B, n = 2, 25
    ids = synth.make_tokens(arch, B, 3 * n, seed=8)
    junk = synth.make_tokens(arch, B, n, seed=9)
    dec = dc.Decoder(arch, "f32", blob, batch=B, chunk_tokens=n)
    ref = run(dec, ids, [n, n, n])
    dec.reset()
    run(dec, ids[:, :2 * n], [n, n])
    snap = dec.export_carry(0)
    run(dec, junk, [n])                      # stream 0 wanders off ...
    dec.import_carry(0, snap)                # ... and rewinds to the checkpoint
    got = run(dec, ids[:, 2 * n:], [n])
    assert bits_equal(got[0], ref[0, 2 * n * dec.spt:])
    dec.close()


def test_snapshot_layouts_must_match():
    arch = synth.REAL_ARCH
    blob = synth.make_weights(arch, 0)
    fused = dc.Decoder(arch, "bf16", blob, batch=8, chunk_tokens=25)
    plain = dc.Decoder(arch, "bf16", blob, batch=8, chunk_tokens=25, flags=dc.DC_NO_FUSE)
    snap = fused.export_carry(0)
    st = dc.dc_carry_import(plain.h, 0, np.resize(snap, dc.dc_carry_bytes(plain.h)))
    assert st == dc.DC_EINVAL                # another ring layout (fused pairs keep wider z contexts)
    assert dc.dc_carry_import(fused.h, 0, snap[:-1]) == dc.DC_EINVAL
    assert dc.dc_carry_import(fused.h, 8, snap) == dc.DC_EINVAL
    bad = snap.copy()
    bad[:8] = 0
    assert dc.dc_carry_import(fused.h, 0, bad) == dc.DC_EINVAL
    assert dc.dc_carry_import(fused.h, 0, snap) == dc.DC_OK
    fused.close()
    plain.close()


SERVE = [
    ("tiny", synth.TINY_ARCH, "f32", 2, 5, 8, 3),
    ("tiny+src", synth.TINY_NSF_ARCH, "f32", 2, 5, 8, 3),
    ("real-bf16-fused", synth.REAL_ARCH, "bf16", 8, 12, 6, 3),
]


@pytest.mark.parametrize("label,arch,dtype,B,S,n,rounds", SERVE, ids=[c[0] for c in SERVE])
def test_more_sessions_than_slots_time_multiplexed(label, arch, dtype, B, S, n, rounds):
    """S sessions served by one state of B < S stream slots (the capacity
    experiment's many sessions on shared weights): each round, every group of
    B sessions is imported into the slots (a new session starts with an
    in-place stream reset), decodes one chunk, and is exported again.  Each
    session's PCM must match the oracle's decode of its own tokens, and (no
    source) the bits of the same sessions decoded side by side without ever
    leaving their slots."""
    blob = synth.make_weights(arch, 4)
    src = arch.get("n_harmonics", 0) > 0
    fpt = arch["frames_per_token"]
    ids = synth.make_tokens(arch, S, rounds * n, seed=11)
    f0 = synth.make_f0(arch, S, rounds * n, seed=11) if src else None
    dec = dc.Decoder(arch, dtype, blob, batch=B, chunk_tokens=n, rng_seed=3)
    snaps, key_slot = [None] * S, [None] * S
    pcm = [[] for _ in range(S)]
    for r in range(rounds):
        for g0 in range(0, S, B):
            group = list(range(g0, min(g0 + B, S)))
            tok = np.zeros((B, n), dtype=np.int32)
            fz = np.full((B, n * fpt), 100.0, dtype=np.float32) if src else None
            for slot, s in enumerate(group):
                if snaps[s] is None:
                    dec.reset_stream(slot)           # a new session: its source key is the slot
                    key_slot[s] = slot
                else:
                    dec.import_carry(slot, snaps[s])
                tok[slot] = ids[s, r * n:(r + 1) * n]
                if src:
                    fz[slot] = f0[s, r * n * fpt:(r + 1) * n * fpt]
            out = (dec.decode(tok, fz) if src else dec.decode(tok)).cpu().numpy()
            for slot, s in enumerate(group):
                pcm[s].append(out[slot])
                snaps[s] = dec.export_carry(slot)
    dec.close()
    got = [np.concatenate(p) for p in pcm]
    worst = 0.0
    for s in range(S):
        if src:
            ref = oracle.decode(arch, dtype, blob, ids[s], f0=f0[s], seed=3, stream=key_slot[s])
        else:
            ref = oracle.decode(arch, dtype, blob, ids[s])
        e, _ = err_stats(got[s], ref)
        worst = max(worst, e)
        assert e <= TOL[dtype], f"{label} session {s}: {e:.3e}"
    say(f"{label}: {S} sessions over {B} slots, {rounds} rounds: worst max-abs/RMS vs oracle {worst:.3e}")
    if not src:
        side = dc.Decoder(arch, dtype, blob, batch=S, chunk_tokens=n)
        ref = run(side, ids, [n] * rounds)
        side.close()
        for s in range(S):
            assert bits_equal(got[s], ref[s]), f"{label} session {s} differs from its uninterrupted decode"


def test_rewound_and_moved_streams_match_the_oracle():
    """A checkpoint taken mid-stream, rewound to after a detour and moved to
    another slot, continues as the oracle's decode of the stream's own tokens."""
    arch = synth.REAL_ARCH
    blob = synth.make_weights(arch, 2)
    B, n = 2, 25
    ids = synth.make_tokens(arch, B, 3 * n, seed=8)
    junk = synth.make_tokens(arch, B, n, seed=9)
    dec = dc.Decoder(arch, "f32", blob, batch=B, chunk_tokens=n)
    head = run(dec, ids[:, :2 * n], [n, n])
    snap = dec.export_carry(0)
    run(dec, junk, [n])                      # both slots wander off
    dec.import_carry(1, snap)                # stream 0's checkpoint continues in slot 1
    tail = run(dec, np.stack([junk[0], ids[0, 2 * n:]]), [n])
    dec.close()
    got = np.concatenate([head[0], tail[1]])
    ref = oracle.decode(arch, "f32", blob, ids[0])
    e, _ = err_stats(got, ref)
    say(f"rewound and moved stream vs oracle: max-abs/RMS {e:.3e}")
    assert e <= TOL["f32"]
