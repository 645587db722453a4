"""Flow-decoder chunk step on the GPU against the fp64 oracle, through the C ABI.

Parity: every chunk's mel frames within 1e-4 (fp32) / 2e-2 (bf16) of the
oracle's, as max-abs-error / RMS; the carry the kernels wrote in place,
read back in Eq. carry's order, within the same bound of the oracle's
concatenated carry (the shadow audit); exact invariants (graph replay equals
direct launches, a stream's result does not depend on the batch, a flush
changes no state, a new turn starts from the prompt alone).
"""
import numpy as np
import pytest

import oracle
from paper_2609_35115_amd import synth
from tests.gpu_common import TOL, bits_equal, err_stats, say

pytestmark = pytest.mark.gpu

TINY = synth.TINY_FLOW_ARCH
SEED = 5


def _flow():
    import torch
    assert torch.cuda.is_available()
    from paper_2609_35115_amd import flow
    return flow


def _prompts(arch, B, P, seed=0):
    return [synth.make_flow_prompt(arch, P, seed=seed, stream=b) for b in range(B)]


def _run_gpu(arch, dtype, blob, B, P, calls, flags=0, prompts=None, mu=None):
    """Prompt every stream, then the calls (frame counts); returns the decoder,
    the per-call mel outputs (numpy [B][n][n_mel]) and the features."""
    flow = _flow()
    dec = flow.FlowDecoder(arch, dtype, blob, B, flags=flags, rng_seed=SEED)
    prompts = prompts or _prompts(arch, B, P)
    for b in range(B):
        dec.prompt(b, *prompts[b])
    total = sum(n for n in calls if n >= arch["f_chunk"]) + arch["f_call"]
    mu = synth.make_flow_mu(arch, B, total) if mu is None else mu
    outs, p = [], 0
    for n in calls:
        outs.append(dec.decode(mu[:, p:p + n]).cpu().numpy())
        if n >= arch["f_chunk"]:
            p += arch["f_chunk"]
    dec.sync()
    return dec, outs, mu, prompts


def _carry_ok(got, want, dtype):
    """The carry audit's bound.  fp32: max-abs-error / RMS as for the output.
    bf16: the carry is stored in bf16, so an element's own rounding is up to
    2^-9 of its magnitude, which against the RMS alone can approach the
    output's 2e-2 for the largest keys; the audit bounds the worst element
    against the largest magnitude and the bulk by the RMS error, both 2e-2."""
    got = np.asarray(got, dtype=np.float64)
    if dtype == "f32":
        e, _ = err_stats(got, want)
        return e <= TOL["f32"], e
    d = np.abs(got - want)
    e1 = d.max() / np.abs(want).max()
    e2 = np.sqrt(np.mean(d ** 2)) / np.sqrt(np.mean(want ** 2))
    return max(e1, e2) <= TOL["bf16"], max(e1, e2)


def _run_oracle(arch, dtype, blob, b, prompt, mu_b, calls):
    s = oracle.FlowStream(arch, dtype, blob, seed=SEED, key=b)
    s.prompt(*prompt)
    outs, p = [], 0
    for n in calls:
        outs.append(s.chunk(mu_b[p:p + n]))
        if n >= arch["f_chunk"]:
            p += arch["f_chunk"]
    return s, outs


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_tiny_chunks_match_oracle(dtype):
    _chunks_match_oracle(TINY, dtype, 5)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_one_head_matches_oracle(dtype):
    """dim = 64 (a single head): the LayerNorm-operand GEMMs take their 4-wave
    shape, whose rows are split over fewer threads."""
    _chunks_match_oracle(dict(TINY, dim=64, heads=1), dtype, 3)


def _chunks_match_oracle(a, dtype, ncalls):
    blob = synth.make_flow_weights(a, 0)
    B, P = 2, a["f_prompt"]
    calls = [a["f_call"]] * ncalls
    say(f"flow tiny dim {a['dim']} {dtype} B={B} calls={calls}")
    dec, outs, mu, prompts = _run_gpu(a, dtype, blob, B, P, calls)
    st = dec.stats()
    assert st["replays"] == ncalls and st["direct"] == 0, st
    worst = 0.0
    for b in range(B):
        s, ref = _run_oracle(a, dtype, blob, b, prompts[b], mu[b], calls)
        for k, (g, r) in enumerate(zip(outs, ref)):
            e, _ = err_stats(g[b], r)
            worst = max(worst, e)
            assert e <= TOL[dtype], f"stream {b} call {k}: {e:.3e}"
        # shadow audit: the carry read back in Eq. carry's order
        for (i, l, c, kv) in [(0, 0, 0, 0), (a["n_steps"] - 1, a["depth"] - 1, 1, 1), (1, 0, 1, 0)]:
            got = dec.carry(b, i, l, c, kv)
            want = s.carry(i, l, c, kv)
            assert got.shape == want.shape
            ok, e = _carry_ok(got, want, dtype)
            e_r15, _ = err_stats(got, want)
            say(f"  carry {(b, i, l, c, kv)}: audit {e:.3e} (max-abs/RMS {e_r15:.3e})")
            assert ok, f"carry {(b, i, l, c, kv)}: {e:.3e}"
    say(f"  worst max-abs/RMS {worst:.3e}")
    dec.close()


def test_partial_calls_and_flush_match_oracle():
    """Calls of other sizes run kernel by kernel: f_chunk frames (no lookahead),
    a call between f_chunk and f_call, and a flush of fewer than f_chunk frames
    that leaves the state unchanged."""
    a = TINY
    blob = synth.make_flow_weights(a, 0)
    fc = a["f_chunk"]
    calls = [a["f_call"], fc, fc + 1, 3, a["f_call"], fc]
    dec, outs, mu, prompts = _run_gpu(a, "f32", blob, 2, 13, calls, prompts=_prompts(a, 2, 13, seed=1))
    st = dec.stats()
    assert st["replays"] == 2 and st["direct"] == 4, st
    for b in range(2):
        _s, ref = _run_oracle(a, "f32", blob, b, prompts[b], mu[b], calls)
        for k, (g, r) in enumerate(zip(outs, ref)):
            e, _ = err_stats(g[b], r)
            assert e <= TOL["f32"], f"stream {b} call {k} (n={calls[k]}): {e:.3e}"
    dec.close()


def test_graph_replay_equals_direct_launches():
    flow = _flow()
    a = TINY
    blob = synth.make_flow_weights(a, 2)
    calls = [a["f_call"]] * 4
    _d1, o1, _mu, _p = _run_gpu(a, "bf16", blob, 3, a["f_prompt"], calls)
    _d2, o2, _mu, _p = _run_gpu(a, "bf16", blob, 3, a["f_prompt"], calls, flags=flow.DC_NO_GRAPH)
    assert _d2.stats()["replays"] == 0
    for x, y in zip(o1, o2):
        assert bits_equal(x, y)


def test_result_does_not_depend_on_the_batch():
    """Stream 0 decoded alone and beside four other streams: bit for bit."""
    a = TINY
    blob = synth.make_flow_weights(a, 3)
    calls = [a["f_call"]] * 3
    prompts = _prompts(a, 5, a["f_prompt"])
    _d5, o5, mu, _p = _run_gpu(a, "f32", blob, 5, a["f_prompt"], calls, prompts=prompts)
    _d1, o1, _mu, _p = _run_gpu(a, "f32", blob, 1, a["f_prompt"], calls, prompts=prompts[:1], mu=mu[:1])
    for x, y in zip(o5, o1):
        assert bits_equal(x[0], y[0])


def test_new_turn_starts_from_the_prompt_alone():
    """A prompt pass in the middle of a stream's life resets its history: the
    next chunks equal those of a fresh state given the same prompt."""
    a = TINY
    blob = synth.make_flow_weights(a, 0)
    flow = _flow()
    prompts = _prompts(a, 1, a["f_prompt"], seed=4)
    dec, _outs, mu, _p = _run_gpu(a, "f32", blob, 1, a["f_prompt"], [a["f_call"]] * 3)
    dec.prompt(0, *prompts[0])
    again = [dec.decode(mu[:, k * a["f_chunk"]:k * a["f_chunk"] + a["f_call"]]).cpu().numpy() for k in range(2)]
    fresh = flow.FlowDecoder(a, "f32", blob, 1, rng_seed=SEED)
    fresh.prompt(0, *prompts[0])
    ref = [fresh.decode(mu[:, k * a["f_chunk"]:k * a["f_chunk"] + a["f_call"]]).cpu().numpy() for k in range(2)]
    for x, y in zip(again, ref):
        assert bits_equal(x, y)
    assert dec.carry(0, 0, 0, 0, 0).shape[0] == a["f_prompt"] + 2 * a["f_chunk"]


def test_extents_follow_the_papers_catalog():
    """The clock quantities of the paper (302, 100, 50, 56) at a small width:
    carried extents 302, 352, 402, 402 (Eq. catalog)."""
    a = dict(TINY, f_prompt=302, f_retained=100, f_chunk=50, f_call=56, n_steps=2, depth=1, dim=64, heads=1,
             mlp=64, n_mel=8, t_dim=8)
    blob = synth.make_flow_weights(a, 0)
    flow = _flow()
    dec = flow.FlowDecoder(a, "bf16", blob, 2, rng_seed=SEED)
    for b in range(2):
        dec.prompt(b, *synth.make_flow_prompt(a, 302, stream=b))
    mu = synth.make_flow_mu(a, 2, 400)
    seen = [dec.carry(1, 0, 0, 0, 0).shape[0]]
    for k in range(3):
        dec.decode(mu[:, 50 * k:50 * k + 56])
        seen.append(dec.carry(1, 1, 0, 1, 1).shape[0])
    assert seen == [302, 352, 402, 402]
    dec.close()


def test_rejects_bad_calls():
    flow = _flow()
    a = TINY
    blob = synth.make_flow_weights(a, 0)
    dec = flow.FlowDecoder(a, "f32", blob, 2, rng_seed=SEED)
    mu = synth.make_flow_mu(a, 2, a["f_call"])
    st = dec.decode(mu, check=False)
    assert dec.stats()["rejected"] == 1                     # no turn yet
    dec.prompt(0, *synth.make_flow_prompt(a, a["f_prompt"]))
    dec.decode(mu, check=False)
    assert dec.stats()["rejected"] == 2                     # stream 1 still has none
    dec.prompt(1, *synth.make_flow_prompt(a, a["f_prompt"], stream=1))
    too_long = synth.make_flow_mu(a, 2, a["f_call"] + 1)
    with pytest.raises(Exception):
        dec.decode(too_long)
    big = synth.make_flow_prompt(a, a["f_prompt"] + 1)
    with pytest.raises(Exception):
        dec.prompt(0, *big)
    out = dec.decode(mu)                                     # still usable
    assert np.isfinite(out.cpu().numpy()).all()
    del st
    dec.close()


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_real_shape_matches_oracle(dtype):
    """The paper-shaped decoder (16 blocks of width 512, 10 solver steps,
    f_call 56, f_chunk 50) with a 64-frame prompt: three calls (extents 64,
    114, 164) against the oracle."""
    a = synth.REAL_FLOW_ARCH
    blob = synth.make_flow_weights(a, 0)
    P = 64
    calls = [a["f_call"]] * 2
    say(f"flow real {dtype} B=1 P={P} calls={calls}")
    dec, outs, mu, prompts = _run_gpu(a, dtype, blob, 1, P, calls)
    s, ref = _run_oracle(a, dtype, blob, 0, prompts[0], mu[0], calls)
    for k, (g, r) in enumerate(zip(outs, ref)):
        e, er = err_stats(g[0], r)
        say(f"  call {k}: max-abs/RMS {e:.3e}, RMS err/RMS {er:.3e}")
        assert e <= TOL[dtype], f"call {k}: {e:.3e}"
    for (i, l, c, kv) in [(9, 15, 0, 1), (0, 7, 1, 0)]:
        ok, e = _carry_ok(dec.carry(0, i, l, c, kv), s.carry(i, l, c, kv), dtype)
        e_r15, _ = err_stats(dec.carry(0, i, l, c, kv), s.carry(i, l, c, kv))
        say(f"  carry {(i, l, c, kv)}: audit {e:.3e} (max-abs/RMS {e_r15:.3e})")
        assert ok, f"carry {(i, l, c, kv)}: {e:.3e}"
    dec.close()


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_real_shape_at_the_papers_extents_matches_oracle(dtype):
    """The paper-shaped decoder at the paper's operating point: a 302-frame
    prompt, then four calls of f_call = 56 frames (50 retained plus 6 of
    lookahead), so the attended extents run 302, 352, 402, 402 and the last two
    calls cut the carry back to H[0:100] || H[ext - 302:ext] (Eq. carry).
    Every call's mel against the oracle, and the carry after the last call
    (the shadow audit) in both metrics."""
    a = synth.REAL_FLOW_ARCH
    blob = synth.make_flow_weights(a, 0)
    P = a["f_prompt"]
    calls = [a["f_call"]] * 4
    say(f"flow real {dtype} B=1 P={P} calls={calls}")
    dec, outs, mu, prompts = _run_gpu(a, dtype, blob, 1, P, calls)
    assert dec.stats()["replays"] == 4
    s, ref = _run_oracle(a, dtype, blob, 0, prompts[0], mu[0], calls)
    assert s.extent == 402
    for k, (g, r) in enumerate(zip(outs, ref)):
        e, er = err_stats(g[0], r)
        say(f"  call {k}: max-abs/RMS {e:.3e}, RMS err/RMS {er:.3e}")
        assert e <= TOL[dtype], f"call {k}: {e:.3e}"
    for (i, l, c, kv) in [(9, 15, 0, 1), (0, 7, 1, 0), (5, 3, 0, 0)]:
        got, want = dec.carry(0, i, l, c, kv), s.carry(i, l, c, kv)
        assert got.shape == want.shape == (402, a["dim"])
        e_r15, _ = err_stats(got, want)
        ok, e = _carry_ok(got, want, dtype)
        say(f"  carry {(i, l, c, kv)}: audit {e:.3e} (max-abs/RMS {e_r15:.3e})")
        assert ok, f"carry {(i, l, c, kv)}: {e:.3e}"
    dec.close()


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_many_rows_take_the_tiled_path_and_match_oracle(dtype):
    """24 streams: a call of 528 rows runs the tiled GEMMs with a standalone
    LayerNorm (calls of at most 512 rows take the skinny GEMMs)."""
    a = TINY
    blob = synth.make_flow_weights(a, 5)
    B = 24
    calls = [a["f_call"]] * 3
    say(f"flow tiny {dtype} B={B} (tiled path)")
    dec, outs, mu, prompts = _run_gpu(a, dtype, blob, B, a["f_prompt"], calls)
    for b in (0, 11, 23):
        _s, ref = _run_oracle(a, dtype, blob, b, prompts[b], mu[b], calls)
        for k, (g, r) in enumerate(zip(outs, ref)):
            e, _ = err_stats(g[b], r)
            assert e <= TOL[dtype], f"stream {b} call {k}: {e:.3e}"
    dec.close()


def test_real_shape_batch20_every_tile_size():
    """20 paper-shaped streams in bf16: 2,240 rows per call, so the MLP-up GEMM
    takes 128 x 128 tiles, the input, QKV, attention-output and MLP-down GEMMs
    128 x 64, and the 80-column output projection 32 x 32."""
    a = synth.REAL_FLOW_ARCH
    blob = synth.make_flow_weights(a, 0)
    B, P = 20, 64
    calls = [a["f_call"]]
    say(f"flow real bf16 B={B} P={P}")
    dec, outs, mu, prompts = _run_gpu(a, "bf16", blob, B, P, calls)
    for b in (0, 19):
        _s, ref = _run_oracle(a, "bf16", blob, b, prompts[b], mu[b], calls)
        e, er = err_stats(outs[0][b], ref[0])
        say(f"  stream {b}: max-abs/RMS {e:.3e}, RMS err/RMS {er:.3e}")
        assert e <= TOL["bf16"], f"stream {b}: {e:.3e}"
    dec.close()


def test_host_pointer_mode_equals_device_mode():
    """DC_HOST_PTRS: host prompts, features and mel (synchronous calls) give the
    bits of the device-pointer path."""
    flow = _flow()
    a = TINY
    blob = synth.make_flow_weights(a, 1)
    calls = [a["f_call"], a["f_call"], a["f_chunk"] - 2]
    _d, dev_out, mu, prompts = _run_gpu(a, "bf16", blob, 2, a["f_prompt"], calls)
    h = flow.FlowDecoder(a, "bf16", blob, 2, flags=flow.DC_HOST_PTRS, rng_seed=SEED)
    for b in range(2):
        h.prompt(b, *prompts[b])
    p = 0
    for k, n in enumerate(calls):
        out = h.decode(np.ascontiguousarray(mu[:, p:p + n]))
        assert isinstance(out, np.ndarray)
        assert bits_equal(out, dev_out[k])
        if n >= a["f_chunk"]:
            p += a["f_chunk"]
    h.close()


@pytest.mark.parametrize("name,streams", [("flow_real_bf16_b16", (0, 15)), ("flow_real_bf16_b128", (0, 127))])
def test_batched_bench_workloads_match_oracle(name, streams):
    """The batched benchmark configurations in the benchmark's launch shapes
    (all streams, a replayed f_call-frame call); sampled streams against the
    oracle.  Prompts of 64 frames keep the oracle's share short (the batch-1
    configurations are the real-shape test above)."""
    w = synth.workload(name)
    a, dtype, B = w["arch"], w["dtype"], w["batch"]
    blob = synth.make_flow_weights(a, 0)
    P = 64
    say(f"{name}: B={B} prompt {P}, one call of {a['f_call']} frames")
    dec, outs, mu, prompts = _run_gpu(a, dtype, blob, B, P, [a["f_call"]])
    assert dec.stats()["replays"] == 1
    for b in streams:
        _s, ref = _run_oracle(a, dtype, blob, b, prompts[b], mu[b], [a["f_call"]])
        e, er = err_stats(outs[0][b], ref[0])
        say(f"  stream {b}: max-abs/RMS {e:.3e}, RMS err/RMS {er:.3e}")
        assert e <= TOL[dtype], f"stream {b}: {e:.3e}"
    dec.close()
