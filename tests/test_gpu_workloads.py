"""Full-size workloads on the GPU, in the launch configuration bench.py times
(chunk shape captured as a graph, device pointers, every stream decoded for
every chunk of the workload).

For every workload:
  * the PCM matches the oracle within the workload's tolerance
    (max-abs-error / RMS, 1e-4 fp32, 2e-2 bf16) on sampled windows: the
    first chunk of a stream, a middle chunk and the last chunk of the first,
    a middle and the last stream -- and with 128 streams one window of every
    stream (the oracle decodes each window from a lead-in longer than the
    decoder's receptive field);
  * the 18-channel head output of the last chunk matches the oracle's head
    tap, with the same metric;
  * the same state re-decoding the whole token stream with direct calls of
    other sizes (up to one offline call of all tokens where the memory of its
    rings allows) reproduces the replayed chunks bit for bit on every stream.
"""
from __future__ import annotations

import numpy as np
import pytest

import oracle
import paper_2609_35115_amd as dc
from paper_2609_35115_amd import synth
from tests.gpu_common import LEAD, TOL, bits_equal, err_stats, oracle_window, say

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

# direct-call sizes of the re-decode (tokens), per workload
REDECODE = {
    "tiny_f32_b1_n8": [64],                      # one offline call
    "real_f32_b1_n25": [500],                    # one offline call
    "real_bf16_b16_n25": [500],                  # one offline call
    "real_bf16_b1_n4": [800],                    # one offline call
    "real_bf16_b128_n25": [100] * 10,            # 100-token calls (offline rings would need ~225 GB)
}


def run_chunked(dec, tok_dev, chunks, n):
    outs = []
    for c in range(chunks):
        outs.append(dec.decode(tok_dev[c]))
    dec.sync()
    return torch.cat(outs, dim=1)


@pytest.mark.parametrize("name", list(synth.WORKLOADS))
def test_workload_parity_and_exactness(name):
    w = synth.workload(name)
    arch, dtype, B, n, chunks = w["arch"], w["dtype"], w["batch"], w["chunk_tokens"], w["chunks"]
    spt = synth.samples_per_token(arch)
    total = chunks * n
    say(f"[{name}] batch {B}, {chunks} chunks x {n} tokens, {dtype}")
    blob = synth.make_weights(arch, 0)
    ids = synth.make_tokens(arch, B, total)
    tok_dev = torch.from_numpy(np.ascontiguousarray(ids.reshape(B, chunks, n).transpose(1, 0, 2))).cuda()

    sizes = REDECODE[name]
    assert sum(sizes) == total
    dec = dc.Decoder(arch, dtype, blob, batch=B, chunk_tokens=n, max_tokens=max(max(sizes), n))
    pcm_dev = run_chunked(dec, tok_dev, chunks, n)
    st = dec.stats()
    assert st["replays"] == chunks and st["direct_shape"] == 0, st
    pcm = pcm_dev.cpu().numpy()
    del pcm_dev
    say(f"[{name}] chunked decode done: {pcm.shape}")

    # re-decode with direct calls of other sizes on the same state
    dec.reset()
    ids_dev = torch.from_numpy(ids).cuda()
    pos = 0
    for m in sizes:
        part = dec.decode(ids_dev[:, pos:pos + m].contiguous())
        dec.sync()
        got = part.cpu().numpy()
        assert bits_equal(got, pcm[:, pos * spt:(pos + m) * spt]), f"tokens [{pos},{pos + m}) differ"
        pos += m
    assert dec.stats()["direct_shape"] == len(sizes) or sizes == [n] * len(sizes)
    say(f"[{name}] re-decode with calls of {sorted(set(sizes))} tokens: bit-exact on all {B} streams")

    # the 18-channel head output of the last chunk (R15's guard against the
    # iSTFT masking an upstream error), read from the state's ring, against
    # the oracle's head tap over the same frames
    fl = synth.frames_per_chunk(arch, 1) * int(np.prod(arch["up_rate"]))   # last-stage frames per token
    s_last = total - n
    for b in sorted({0, B - 1}):
        got = dec.tap("head", b, s_last * fl, n * fl)
        s0 = max(0, s_last - LEAD)
        _pcm, ref = oracle.decode(arch, dtype, blob, ids[b, s0:total], tap="head")
        emax, erms = err_stats(got, ref[(s_last - s0) * fl:])
        say(f"[{name}] stream {b} head tap, tokens [{s_last},{total}): max-abs-err/RMS {emax:.3e} rms {erms:.3e}")
        assert emax <= TOL[dtype], f"stream {b} head tap: {emax:.3e} > {TOL[dtype]}"
    dec.close()

    # oracle on sampled windows: the first, a middle and the last chunk of the
    # first, a middle and the last stream; with many streams, every stream on
    # one window (the last chunk for every fourth stream)
    if B >= 64:
        last = (chunks - 1) * n
        plan = [(b, last if b % 4 == 0 else (b % chunks) * n) for b in range(B)]
    else:
        plan = [(b, s) for b in sorted({0, B // 2, B - 1}) for s in sorted({0, (chunks // 2) * n, (chunks - 1) * n})]
    worst = 0.0
    for b, s in plan:
        ref = oracle_window(arch, dtype, blob, ids[b], s, s + n)
        got = pcm[b, s * spt:(s + n) * spt]
        emax, erms = err_stats(got, ref)
        worst = max(worst, emax)
        say(f"[{name}] stream {b} tokens [{s},{s + n}): max-abs-err/RMS {emax:.3e} rms {erms:.3e}")
        assert emax <= TOL[dtype], f"stream {b} window {s}: {emax:.3e} > {TOL[dtype]}"
    say(f"[{name}] worst max-abs-err/RMS {worst:.3e} over {len(plan)} windows (tolerance {TOL[dtype]})")
