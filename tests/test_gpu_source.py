"""The harmonic-plus-noise excitation source on the GPU, through the C ABI.

The source is the stochastic input of the paper's vocoder (Design, clause
(iii): a harmonic generator drawing device randomness on every call, admitted
to replay because its generator is counter-based).  Its draws and phases here
depend only on each stream's samples since its start, so:
  * the PCM matches the oracle (which computes the source from the same
    Philox4x64-10 definition, independently) within the workload tolerance,
    and the source samples themselves match the oracle's;
  * chunked equals offline, and graph replay equals direct launches, bit for
    bit;
  * a stream reset mid-run equals a fresh stream bit for bit.
The oracle decodes whole streams here: the source's phase never forgets its
start, so a window cannot be decoded from a lead-in.
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

TINY = synth.TINY_NSF_ARCH
REAL = synth.REAL_NSF_ARCH
SEED = 11


def f0_of(arch, ids_shape, seed=0):
    return synth.make_f0(arch, ids_shape[0], ids_shape[1], seed=seed)


def decode_chunks(dec, ids, f0, sizes):
    fpt = dec.arch["frames_per_token"]
    outs, pos = [], 0
    for n in sizes:
        outs.append(dec.decode(ids[:, pos:pos + n], f0[:, pos * fpt:(pos + n) * fpt]))
        pos += n
    dec.sync()
    return np.concatenate([o if isinstance(o, np.ndarray) else o.cpu().numpy() for o in outs], axis=1)


def check_oracle(arch, dtype, blob, ids, f0, pcm, label):
    worst = 0.0
    for b in range(ids.shape[0]):
        ref = oracle.decode(arch, dtype, blob, ids[b], f0=f0[b], seed=SEED, stream=b)
        emax, erms = err_stats(pcm[b, :ref.size], ref)
        worst = max(worst, emax)
        say(f"{label} stream {b}: max-abs-err/RMS {emax:.3e}, rms-err/RMS {erms:.3e}")
        assert emax <= TOL[dtype], f"{label} stream {b}: {emax:.3e} > {TOL[dtype]}"
    return worst


def test_tiny_source_matches_oracle_and_offline():
    blob = synth.make_weights(TINY, 0)
    ids = synth.make_tokens(TINY, 2, 40)
    f0 = f0_of(TINY, ids.shape)
    say("tiny f32 with source, B=2: chunks of 8, 8, 5, 8, 8, 3 tokens")
    dec = dc.Decoder(TINY, "f32", blob, batch=2, chunk_tokens=8, max_tokens=40, rng_seed=SEED)
    pcm = decode_chunks(dec, ids, f0, [8, 8, 5, 8, 8, 3])
    st = dec.stats()
    assert st["replays"] == 4 and st["direct_shape"] == 2 and st["staged_f0"] == 6, st
    check_oracle(TINY, "f32", blob, ids, f0, pcm, "tiny+src")
    # the source samples of the last call against the oracle's
    last = ids.shape[1] * synth.frames_per_chunk(TINY, 1) * int(np.prod(TINY["up_rate"]))
    nfr = 3 * int(np.prod(TINY["up_rate"]))
    for b in range(2):
        got = dec.tap("src", b, last - nfr, nfr)
        _, ref = oracle.decode(TINY, "f32", blob, ids[b], tap="src", f0=f0[b], seed=SEED, stream=b)
        err = np.abs(got - ref[-nfr:]).max()
        say(f"tiny src tap stream {b}: max abs err {err:.2e}")
        assert err < 2e-5
    dec.reset()
    off = decode_chunks(dec, ids, f0, [40])
    assert bits_equal(off, pcm), "chunked != offline with the source"
    dec.close()


def test_real_f32_source_matches_oracle():
    blob = synth.make_weights(REAL, 1)
    ids = synth.make_tokens(REAL, 1, 50, seed=1)
    f0 = f0_of(REAL, ids.shape, seed=1)
    dec = dc.Decoder(REAL, "f32", blob, batch=1, chunk_tokens=25, rng_seed=SEED)
    pcm = decode_chunks(dec, ids, f0, [25, 25])
    check_oracle(REAL, "f32", blob, ids, f0, pcm, "real f32+src")
    dec.close()


@pytest.mark.parametrize("batch", [3, 8])
def test_real_bf16_source_matches_oracle_and_offline(batch):
    blob = synth.make_weights(REAL, 0)
    ids = synth.make_tokens(REAL, batch, 50)
    f0 = f0_of(REAL, ids.shape)
    dec = dc.Decoder(REAL, "bf16", blob, batch=batch, chunk_tokens=25, max_tokens=50, rng_seed=SEED)
    pcm = decode_chunks(dec, ids, f0, [25, 25])
    check_oracle(REAL, "bf16", blob, ids[:2], f0[:2], pcm[:2], f"real bf16+src B={batch}")
    dec.reset()
    off = decode_chunks(dec, ids, f0, [50])
    assert bits_equal(off, pcm), "chunked != offline with the source"
    dec.close()


def test_replay_equals_direct_and_reset_stream_equals_fresh():
    blob = synth.make_weights(TINY, 3)
    ids = synth.make_tokens(TINY, 3, 24, seed=3)
    f0 = f0_of(TINY, ids.shape, seed=3)
    a = dc.Decoder(TINY, "f32", blob, batch=3, chunk_tokens=8, rng_seed=SEED)
    b = dc.Decoder(TINY, "f32", blob, batch=3, chunk_tokens=8, flags=dc.DC_NO_GRAPH, rng_seed=SEED)
    pa = decode_chunks(a, ids, f0, [8, 8, 8])
    pb = decode_chunks(b, ids, f0, [8, 8, 8])
    assert a.stats()["replays"] == 3 and b.stats()["direct_nograph"] == 3
    assert bits_equal(pa, pb), "replay != direct with the source"
    # stream 1 restarts: its next chunk equals a fresh state's first chunk
    a.reset_stream(1)
    more_ids = synth.make_tokens(TINY, 3, 8, seed=9)
    more_f0 = f0_of(TINY, more_ids.shape, seed=9)
    again = decode_chunks(a, more_ids, more_f0, [8])
    fresh = dc.Decoder(TINY, "f32", blob, batch=3, chunk_tokens=8, rng_seed=SEED)
    first = decode_chunks(fresh, more_ids, more_f0, [8])
    assert bits_equal(again[1], first[1]), "reset stream != fresh stream"
    assert not bits_equal(again[0], first[0])      # the others keep their carry
    for d in (a, b, fresh):
        d.close()


def test_source_admission_fails_closed():
    blob = synth.make_weights(TINY, 0)
    ids = synth.make_tokens(TINY, 1, 8)
    f0 = f0_of(TINY, ids.shape)
    dec = dc.Decoder(TINY, "f32", blob, batch=1, chunk_tokens=8, rng_seed=SEED)
    tok = torch.from_numpy(ids).cuda()
    out = torch.empty((1, 8 * dec.spt), device="cuda")
    assert dc.dc_decode_chunk(dec.h, tok, 8, out) == dc.DC_EINVAL       # needs f0
    assert dc.dc_decode_chunk_f0(dec.h, tok, None, 8, out) == dc.DC_EINVAL
    assert dec.stats()["calls"] == 0 and dec.stats()["rejected"] == 2
    assert dc.dc_f0_buffer(dec.h)
    f0d = torch.from_numpy(f0).cuda()
    torch.cuda.synchronize()
    assert dc.dc_decode_chunk_f0(dec.h, tok, f0d, 8, out) == dc.DC_OK
    dec.sync()
    assert dec.stats()["staged_f0"] == 1
    plain = dc.Decoder(synth.TINY_ARCH, "f32", synth.make_weights(synth.TINY_ARCH), batch=1, chunk_tokens=8)
    assert dc.dc_decode_chunk_f0(plain.h, tok, f0d, 8, out) == dc.DC_EINVAL
    assert dc.dc_f0_buffer(plain.h) is None
    # host-pointer mode
    host = dc.Decoder(TINY, "f32", blob, batch=1, chunk_tokens=8, flags=dc.DC_HOST_PTRS, rng_seed=SEED)
    ph = host.decode(ids, f0)
    dec.reset()
    pd = decode_chunks(dec, ids, f0, [8])
    assert bits_equal(ph, pd)
    for d in (dec, plain, host):
        d.close()


def test_nsf_workload_full_size():
    """real_bf16_b16_n25_nsf in the launch configuration bench.py times: 20
    replayed chunks, then 100-token direct calls reproduce them bit for bit;
    streams 0 and 15 against the oracle over all 500 tokens."""
    name = "real_bf16_b16_n25_nsf"
    w = synth.workload(name)
    arch, dtype, B, n, chunks = w["arch"], w["dtype"], w["batch"], w["chunk_tokens"], w["chunks"]
    total = n * chunks
    blob = synth.make_weights(arch, 0)
    ids = synth.make_tokens(arch, B, total)
    f0 = synth.make_f0(arch, B, total)
    dec = dc.Decoder(arch, dtype, blob, batch=B, chunk_tokens=n, max_tokens=100, rng_seed=SEED)
    pcm = decode_chunks(dec, ids, f0, [n] * chunks)
    assert dec.stats()["replays"] == chunks
    say(f"[{name}] chunked decode done: {pcm.shape}")
    dec.reset()
    again = decode_chunks(dec, ids, f0, [100] * (total // 100))
    assert bits_equal(again, pcm), "100-token calls != 25-token replays"
    dec.close()
    for b in (0, B - 1):
        ref = oracle.decode(arch, dtype, blob, ids[b], f0=f0[b], seed=SEED, stream=b)
        emax, erms = err_stats(pcm[b], ref)
        say(f"[{name}] stream {b}, all {total} tokens: max-abs-err/RMS {emax:.3e} rms {erms:.3e}")
        assert emax <= TOL[dtype]
