"""GPU parity of the C-ABI decode step against the oracle, and the exactness
properties of the streaming form (chunked == offline, replay == direct, tile
shape, batch independence, reset), on small inputs."""
from __future__ import annotations

import numpy as np
import pytest

import oracle
import paper_2609_35115_amd as dc
from paper_2609_35115_amd import synth
from tests.gpu_common import TOL, bits_equal, err_stats, oracle_window, say

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

TINY = synth.TINY_ARCH
REAL = synth.REAL_ARCH


def decode_chunks(dec, ids, sizes):
    outs, pos = [], 0
    for n in sizes:
        outs.append(dec.decode(ids[:, pos:pos + n]))
        pos += n
    dec.sync()
    return np.concatenate([o.cpu().numpy() for o in outs], axis=1)


def check_oracle(arch, dtype, blob, ids, pcm, label):
    spt = synth.samples_per_token(arch)
    for b in range(ids.shape[0]):
        ref = oracle.decode(arch, dtype, blob, ids[b])
        emax, erms = err_stats(pcm[b, :ref.size], ref)
        say(f"{label} stream {b}: max-abs-err/RMS {emax:.3e}, rms-err/RMS {erms:.3e}")
        assert emax <= TOL[dtype], f"{label} stream {b}: {emax:.3e} > {TOL[dtype]}"
    assert pcm.shape[1] == ids.shape[1] * spt


def test_tiny_f32_matches_oracle_chunked():
    blob = synth.make_weights(TINY, 0)
    ids = synth.make_tokens(TINY, 2, 64)
    say("tiny f32 B=2: 8 chunks of 8 tokens")
    dec = dc.Decoder(TINY, "f32", blob, batch=2, chunk_tokens=8)
    pcm = decode_chunks(dec, ids, [8] * 8)
    st = dec.stats()
    assert st["replays"] == 8 and st["direct_shape"] == 0
    check_oracle(TINY, "f32", blob, ids, pcm, "tiny f32")
    dec.close()


def test_tiny_taps_match_oracle_intermediates():
    """Every carried ring holds the oracle's intermediate for the frames it keeps."""
    blob = synth.make_weights(TINY, 0)
    ids = synth.make_tokens(TINY, 1, 24)
    dec = dc.Decoder(TINY, "f32", blob, batch=1, chunk_tokens=8)
    decode_chunks(dec, ids, [8, 8, 8])
    names = ["embed", "pre0", "pre3", "s0.y", "s0.rb0.h0", "s0.rb0.z0", "s0.x", "s1.y", "s2.x", "head"]
    for name in names:
        _, ref = oracle.decode(TINY, "f32", blob, ids[0], tap=name)
        if ".h" in name:
            ref = np.where(ref >= 0, ref, TINY["lrelu_slope"] * ref)
        frames = ref.shape[0]
        last = frames // 3          # frames of the last call
        got = dec.tap(name, 0, frames - last, last)
        err = np.abs(got - ref[frames - last:]).max() / (np.abs(ref).max() + 1e-30)
        say(f"tap {name}: rel max err {err:.3e}")
        assert err < 1e-5, name
    dec.close()


@pytest.mark.parametrize("arch_name,dtype,sizes", [
    ("tiny", "f32", [8, 8, 3, 8, 1, 8]),
    ("real", "f32", [4, 4, 1, 4]),
    ("real", "bf16", [4, 4, 3, 4]),
])
def test_chunked_equals_offline_bit_exact(arch_name, dtype, sizes):
    arch = TINY if arch_name == "tiny" else REAL
    blob = synth.make_weights(arch, 0)
    total = sum(sizes)
    ids = synth.make_tokens(arch, 2, total)
    say(f"chunked vs offline {arch_name} {dtype} sizes {sizes}")
    dec = dc.Decoder(arch, dtype, blob, batch=2, chunk_tokens=sizes[0], max_tokens=total)
    chunked = decode_chunks(dec, ids, sizes)
    dec.reset()
    offline = decode_chunks(dec, ids, [total])
    assert bits_equal(chunked, offline)
    dec.close()


@pytest.mark.parametrize("arch_name,dtype", [("tiny", "f32"), ("real", "bf16")])
def test_graph_replay_equals_direct_launch(arch_name, dtype):
    arch = TINY if arch_name == "tiny" else REAL
    n = 8 if arch_name == "tiny" else 4
    blob = synth.make_weights(arch, 1)
    ids = synth.make_tokens(arch, 2, 3 * n)
    a = dc.Decoder(arch, dtype, blob, batch=2, chunk_tokens=n)
    b = dc.Decoder(arch, dtype, blob, batch=2, chunk_tokens=n, flags=dc.DC_NO_GRAPH)
    pa = decode_chunks(a, ids, [n] * 3)
    pb = decode_chunks(b, ids, [n] * 3)
    assert a.stats()["replays"] == 3 and b.stats()["direct_nograph"] == 3
    assert bits_equal(pa, pb)
    a.close()
    b.close()


# Forced tile shapes (1-based tile_variant) that share the arithmetic -- K
# partitions across waves and channel block -- and fit every layer of the
# case: their results must be identical.
TILE_GROUPS = {
    ("tiny", "f32", "unsplit"): [7, 10, 13],     # 32x32, 64x64, 128x64; unsplit K, 32-channel blocks
    ("real", "f32", "kch4"): [1, 4, 6],          # 16x16, 16x32, 32x32; K in 4 partitions, 64-channel blocks
    ("real", "f32", "kch8"): [2, 5, 28],         # 16x16, 16x32, 32x32; K in 4 partitions, 128-channel blocks
    ("real", "bf16", "unsplit"): [8, 9, 11,      # 32x32, 32x64, 64x64; unsplit K, 128-channel blocks
                                  21, 22, 25, 26, 27],   # the same with weights through the LDS ring
    ("real", "bf16", "kch2"): [7, 10, 13, 29],   # 32x32, 64x64, 128x64, 128x32; 64-channel blocks
}


@pytest.mark.parametrize("arch_name,dtype,group", list(TILE_GROUPS))
def test_tile_shape_does_not_change_results(arch_name, dtype, group):
    arch = TINY if arch_name == "tiny" else REAL
    n = 8 if arch_name == "tiny" else 3
    blob = synth.make_weights(arch, 2)
    ids = synth.make_tokens(arch, 1, 2 * n)
    variants = TILE_GROUPS[(arch_name, dtype, group)]
    ref = None
    for v in variants:
        dec = dc.Decoder(arch, dtype, blob, batch=1, chunk_tokens=n, tile_variant=v)
        pcm = decode_chunks(dec, ids, [n, n])
        dec.close()
        if ref is None:
            ref = pcm
        else:
            assert bits_equal(pcm, ref), f"tile variant {v} differs from {variants[0]}"


def test_real_f32_matches_oracle():
    blob = synth.make_weights(REAL, 0)
    ids = synth.make_tokens(REAL, 1, 50)
    say("real f32 B=1: 2 chunks of 25 tokens")
    dec = dc.Decoder(REAL, "f32", blob, batch=1, chunk_tokens=25)
    pcm = decode_chunks(dec, ids, [25, 25])
    check_oracle(REAL, "f32", blob, ids, pcm, "real f32")
    dec.close()


def test_real_bf16_matches_oracle():
    blob = synth.make_weights(REAL, 0)
    ids = synth.make_tokens(REAL, 3, 50)
    say("real bf16 B=3: 2 chunks of 25 tokens")
    dec = dc.Decoder(REAL, "bf16", blob, batch=3, chunk_tokens=25)
    pcm = decode_chunks(dec, ids, [25, 25])
    check_oracle(REAL, "bf16", blob, ids, pcm, "real bf16")
    dec.close()


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_stream_in_batch_equals_stream_alone(dtype):
    blob = synth.make_weights(REAL, 0)
    ids = synth.make_tokens(REAL, 3, 8)
    big = dc.Decoder(REAL, dtype, blob, batch=3, chunk_tokens=4, tile_variant=11)
    pb = decode_chunks(big, ids, [4, 4])
    big.close()
    one = dc.Decoder(REAL, dtype, blob, batch=1, chunk_tokens=4, tile_variant=8)
    p1 = decode_chunks(one, ids[2:3], [4, 4])
    one.close()
    assert bits_equal(pb[2:3], p1)


# Automatic tile choice (tile_variant 0): the arithmetic depends on the layer,
# the dtype and the batch class only.  A fresh state whose chunk holds the
# whole utterance decodes it to the bits of a chunked decode, and a stream's
# bits do not depend on the batch it shares (within one class).
@pytest.mark.parametrize("dtype,batch", [("f32", 1), ("bf16", 1), ("bf16", 16)])
def test_whole_utterance_state_equals_chunked_automatic_tiles(dtype, batch):
    blob = synth.make_weights(REAL, 0)
    ids = synth.make_tokens(REAL, batch, 100)
    say(f"real {dtype} B={batch}: 4 chunks of 25 vs a state with chunk_tokens=100")
    a = dc.Decoder(REAL, dtype, blob, batch=batch, chunk_tokens=25)
    pa = decode_chunks(a, ids, [25] * 4)
    assert a.stats()["replays"] == 4
    a.close()
    b = dc.Decoder(REAL, dtype, blob, batch=batch, chunk_tokens=100)
    pb = decode_chunks(b, ids, [100])
    assert b.stats()["replays"] == 1
    b.close()
    assert bits_equal(pa, pb)


# (batch 7 is the largest of the streaming class, batch 8 the smallest of the
# batched one)
@pytest.mark.parametrize("dtype,big,small", [("f32", 3, 1), ("bf16", 3, 1), ("bf16", 7, 1), ("bf16", 16, 8),
                                             ("f32", 12, 8)])
def test_stream_bits_independent_of_batch_within_class(dtype, big, small):
    blob = synth.make_weights(REAL, 0)
    ids = synth.make_tokens(REAL, big, 8)
    say(f"real {dtype}: batch {big} vs batch {small}, automatic tiles")
    a = dc.Decoder(REAL, dtype, blob, batch=big, chunk_tokens=4)
    pa = decode_chunks(a, ids, [4, 4])
    a.close()
    b = dc.Decoder(REAL, dtype, blob, batch=small, chunk_tokens=8)
    pb = decode_chunks(b, ids[big - small:], [8])
    b.close()
    assert bits_equal(pa[big - small:], pb)


def test_reset_and_reset_stream_equal_fresh_state():
    blob = synth.make_weights(TINY, 0)
    ids = synth.make_tokens(TINY, 2, 24)
    dec = dc.Decoder(TINY, "f32", blob, batch=2, chunk_tokens=8)
    fresh = decode_chunks(dec, ids, [8, 8])
    decode_chunks(dec, ids, [8])             # advance, then reset
    dec.reset()
    again = decode_chunks(dec, ids, [8, 8])
    assert bits_equal(fresh, again)
    # stream 1 reset mid-way behaves like a fresh stream; stream 0 is untouched
    dec.reset()
    first = decode_chunks(dec, ids, [8])
    dec.reset_stream(1)
    second = decode_chunks(dec, ids[:, :8], [8])
    assert bits_equal(second[1], first[1])
    cont = dc.Decoder(TINY, "f32", blob, batch=2, chunk_tokens=8)
    ref = decode_chunks(cont, np.concatenate([ids[:, :8], ids[:, :8]], axis=1), [8, 8])
    assert bits_equal(second[0], ref[0, 512:])
    cont.close()
    dec.close()


def test_admission_fails_closed_and_leaves_state_unchanged():
    blob = synth.make_weights(TINY, 0)
    ids = synth.make_tokens(TINY, 1, 24)
    dec = dc.Decoder(TINY, "f32", blob, batch=1, chunk_tokens=8, max_tokens=8)
    a = dec.decode(ids[:, :8])
    tok = torch.from_numpy(ids[:, 8:16].copy()).cuda()
    out = torch.empty((1, 16 * 64), device="cuda")
    assert dc.dc_decode_chunk(dec.h, tok, 16, out) == dc.DC_ERANGE
    assert dc.dc_decode_chunk(dec.h, tok, 0, out) == dc.DC_EINVAL
    assert dc.dc_decode_chunk(dec.h, tok, -3, out) == dc.DC_EINVAL
    assert dc.dc_decode_chunk(dec.h, None, 8, out) == dc.DC_EINVAL
    assert dec.stats()["rejected"] == 4
    b = dec.decode(ids[:, 8:16])
    dec.sync()
    ref = dc.Decoder(TINY, "f32", blob, batch=1, chunk_tokens=8)
    r = decode_chunks(ref, ids, [8, 8])
    ref.close()
    got = np.concatenate([a.cpu().numpy(), b.cpu().numpy()], axis=1)
    assert bits_equal(got, r)
    dec.close()


def test_out_of_range_ids():
    blob = synth.make_weights(TINY, 0)
    ids = synth.make_tokens(TINY, 1, 8)
    bad = ids.copy()
    bad[0, 3] = TINY["vocab"]
    # host pointers: refused before any launch, state unchanged
    h = dc.Decoder(TINY, "f32", blob, batch=1, chunk_tokens=8, flags=dc.DC_HOST_PTRS)
    with pytest.raises(dc.DcError) as e:
        h.decode(bad)
    assert e.value.status == dc.DC_ERANGE
    got = h.decode(ids)
    ref = oracle.decode(TINY, "f32", blob, ids[0])
    assert err_stats(got[0], ref)[0] <= 1e-4
    h.close()
    # device pointers: the kernel raises the flag, dc_sync reports it, state poisoned until reset
    d = dc.Decoder(TINY, "f32", blob, batch=1, chunk_tokens=8)
    d.decode(bad)
    assert dc.dc_sync(d.h) == dc.DC_ERANGE
    out = torch.empty((1, 8 * 64), device="cuda")
    tok = torch.from_numpy(ids).cuda()
    assert dc.dc_decode_chunk(d.h, tok, 8, out) == dc.DC_ESTATE
    d.reset()
    p = decode_chunks(d, ids, [8])
    assert err_stats(p[0], ref)[0] <= 1e-4
    d.close()


def test_binary16_overflow_raises_the_flag():
    """A bf16 state keeps its residual stream in binary16: with the embedding
    scaled far past that range, the stores raise the device flag (dc_sync:
    DC_ERANGE naming the overflow, the state poisoned until dc_reset), where a
    normal decode raises nothing; an fp32 state has no such limit."""
    blob = synth.make_weights(TINY, 0)
    big = blob.copy()
    synth.split_weights(TINY, big)["emb"][...] *= 1.0e6
    ids = synth.make_tokens(TINY, 1, 8)
    ok = dc.Decoder(TINY, "bf16", blob, batch=1, chunk_tokens=8)
    ok.decode(ids)
    assert dc.dc_sync(ok.h) == dc.DC_OK
    ok.close()
    d = dc.Decoder(TINY, "bf16", big, batch=1, chunk_tokens=8)
    d.decode(ids)
    assert dc.dc_sync(d.h) == dc.DC_ERANGE
    assert "binary16" in dc.dc_last_error(d.h)
    out = torch.empty((1, 8 * 64), device="cuda")
    assert dc.dc_decode_chunk(d.h, torch.from_numpy(ids).cuda(), 8, out) == dc.DC_ESTATE
    d.reset()
    assert dc.dc_sync(d.h) == dc.DC_OK
    d.close()
    f = dc.Decoder(TINY, "f32", big, batch=1, chunk_tokens=8)
    f.decode(ids)
    assert dc.dc_sync(f.h) == dc.DC_OK
    f.close()


# The last branch's last conv of the last stage writes the stage output x, the
# last binary16 store before the head (whose outputs are fp32): planted there,
# only that launch can raise the flag.
@pytest.mark.parametrize("planted,flags,tv,kernel", [
    ("s2.rb2.d2.W2", 0, 0, "pair_kernel"),                 # the fused branch-mean pair
    ("s2.rb2.d2.W2", dc.DC_NO_FUSE, 0, "conv_kernel"),     # the same conv unfused
    ("s2.rb2.d2.W2", dc.DC_NO_FUSE, 27, "wconv_kernel"),   # unfused, 64x64 tiles, weights through the LDS ring
    ("s2.up.W", 0, 0, None),                               # the transposed conv's y (and what follows it)
])
def test_binary16_overflow_raises_the_flag_in_the_batched_kernels(planted, flags, tv, kernel):
    """The batched class (batch >= 8) stores the residual stream through other
    kernels than batch 1 does: a weight scaled far past binary16's range makes
    the stores of its layer raise the flag, and the unplanted weights raise
    nothing."""
    B, n = 8, 4
    blob = synth.make_weights(REAL, 0)
    ids = synth.make_tokens(REAL, B, n)
    ok = dc.Decoder(REAL, "bf16", blob, batch=B, chunk_tokens=n, flags=flags, tile_variant=tv)
    ok.decode(ids)
    assert dc.dc_sync(ok.h) == dc.DC_OK
    ok.close()
    big = blob.copy()
    synth.split_weights(REAL, big)[planted][...] *= 1.0e6
    d = dc.Decoder(REAL, "bf16", big, batch=B, chunk_tokens=n, flags=flags, tile_variant=tv)
    named = [f"{l['name']}: {l['kernel']}" for l in d.layers()
             if l['name'].startswith("s2.") and ("mean" in l['name'] or ".up" in l['name'])]
    say(f"binary16 flag: {planted} x 1e6, flags {flags}, tile variant {tv}; {named}")
    if kernel:   # the planted conv runs in the kernel this case is for
        assert any(".mean" in x and f"dc::{kernel}<" in x for x in named), named
    d.decode(ids)
    assert dc.dc_sync(d.h) == dc.DC_ERANGE
    assert "binary16" in dc.dc_last_error(d.h)
    d.reset()
    assert dc.dc_sync(d.h) == dc.DC_OK
    d.close()


def test_fixed_addresses_and_aliasing():
    """Buffers keep their addresses across calls and resets; passing them
    aliases the call (no staging copy) with identical output."""
    blob = synth.make_weights(TINY, 0)
    ids = synth.make_tokens(TINY, 1, 16)
    dec = dc.Decoder(TINY, "f32", blob, batch=1, chunk_tokens=8)
    tb, ab = dc.dc_token_buffer(dec.h), dc.dc_audio_buffer(dec.h)
    staged = dec.decode(ids[:, :8]).cpu().numpy()
    dec.sync()
    st0 = dec.stats()
    assert st0["staged_tokens"] == 1 and st0["staged_audio"] == 1
    dec.reset()
    tok = torch.from_numpy(ids[:, :8].copy()).cuda()
    torch.cuda.synchronize()
    _hip_copy(tb, tok.data_ptr(), 8 * 4)
    assert dc.dc_decode_chunk(dec.h, _Addr(tb), 8, _Addr(ab)) == dc.DC_OK
    dec.sync()
    st1 = dec.stats()
    assert st1["staged_tokens"] == st0["staged_tokens"] and st1["staged_audio"] == st0["staged_audio"]
    out = np.empty(8 * 64, dtype=np.float32)
    _hip_copy(out.ctypes.data, ab, out.nbytes)
    assert bits_equal(out, staged[0])
    assert dc.dc_token_buffer(dec.h) == tb and dc.dc_audio_buffer(dec.h) == ab
    dec.close()


class _Addr:
    """A raw address passed through the binding's pointer marshalling."""

    def __init__(self, addr):
        self.addr = addr

    def data_ptr(self):
        return self.addr


def _hip_copy(dst: int, src: int, nbytes: int):
    import ctypes
    hip = ctypes.CDLL("libamdhip64.so")
    hip.hipMemcpy.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_size_t, ctypes.c_int]
    assert hip.hipMemcpy(dst, src, nbytes, 4) == 0   # hipMemcpyDefault
