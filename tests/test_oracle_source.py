"""Pins of the oracle's harmonic-plus-noise excitation source (CPU only).

The source is the stochastic input of the paper's vocoder (Design, clause
(iii): a harmonic generator that draws device randomness on every call, with
a device-resident sinusoid frequency table and harmonic multiplier).  The
paper prints no formula for it, so it is pinned by
  * numpy's Philox4x64-10 (the library generator of the same published
    definition) for the counter-based draws and their counter layout,
  * Box-Muller special cases and the normal distribution of the draws,
  * closed forms of the sinusoids: constant f0, and piecewise-constant f0
    against a phase summed sample by sample with numpy,
  * where the source enters the decoder, from planted weights.
"""
import math

import numpy as np
import pytest
from scipy import stats

import oracle
from paper_2609_35115_amd import synth

TINY_SRC = dict(synth.TINY_NSF_ARCH)
SPF = synth.TINY_NSF_ARCH["hop"] * math.prod(synth.TINY_NSF_ARCH["up_rate"])   # samples per f0 frame


def np_philox(ctr, key):
    """Philox4x64-10 block of counter ctr from numpy (its bit generator
    advances the 256-bit counter before each block, so it starts at ctr - 1)."""
    v = sum(int(x) << (64 * i) for i, x in enumerate(ctr))
    v = (v - 1) % (1 << 256)
    c = np.array([(v >> (64 * i)) & ((1 << 64) - 1) for i in range(4)], dtype=np.uint64)
    bg = np.random.Philox(counter=c, key=np.array(key, dtype=np.uint64))
    return bg.random_raw(4)


@pytest.mark.parametrize("ctr,key", [
    ((1, 0, 0, 0), (0, 0)),
    ((7, 3, 1, 0), (12345, 678)),
    ((2 ** 40 + 5, 2, 0, 9), (2 ** 63 + 11, 2 ** 62 - 1)),
    ((123456789, 0, 1, 0), (0, 127)),
    ((0, 0, 0, 0), (1, 2)),
    ((0, 3, 1, 0), (2 ** 64 - 1, 0)),
])
def test_philox_matches_numpy(ctr, key):
    assert np.array_equal(oracle.philox4x64(ctr, key), np_philox(ctr, key))


def test_u01_range_and_ends():
    assert oracle.u01(0) == 0.5 * 2.0 ** -53
    assert oracle.u01(2 ** 64 - 1) == 1.0 - 2.0 ** -54
    assert oracle.u01(1 << 63) == 0.5 + 0.5 * 2.0 ** -53


def test_box_muller_special_cases():
    g0, g1 = oracle.box_muller(math.exp(-0.5), 0.25)      # radius 1, angle pi/2
    assert abs(g0) < 1e-15 and abs(g1 - 1.0) < 1e-15
    g0, g1 = oracle.box_muller(math.exp(-2.0), 0.5)       # radius 2, angle pi
    assert abs(g0 + 2.0) < 1e-15 and abs(g1) < 1e-15
    g0, g1 = oracle.box_muller(math.exp(-4.5), 0.0)       # radius 3, angle 0
    assert abs(g0 - 3.0) < 1e-14 and g1 == 0.0


def source_of(arch, f0, merge, merge_b=0.0, seed=5, stream=2):
    return oracle.source(arch, np.asarray(f0, dtype=np.float64), seed, stream, merge, merge_b)


def test_unvoiced_source_is_gaussian_noise_on_the_documented_counters():
    """f0 = 0: no sinusoid, noise of amplitude A/3; merging one harmonic h
    recovers its noise, which must be lane h % 4 of the Box-Muller pairs of
    counter (t, h // 4, 0, 0)."""
    arch = TINY_SRC
    A = arch["sine_amp"]
    H1 = arch["n_harmonics"] + 1
    F = 40
    f0 = np.zeros(F)
    seed, stream = 5, 2
    draws = []
    for h in range(H1):
        merge = np.zeros(H1)
        merge[h] = 1.0
        src = source_of(arch, f0, merge, seed=seed, stream=stream)
        noise = np.arctanh(src) / (A / 3.0)
        draws.append(noise)
        for t in (0, 1, 63, 64, 1000, F * SPF - 1):
            x = np_philox((t, h // 4, 0, 0), (seed, stream))
            pair = h % 4 // 2
            g = oracle.box_muller(oracle.u01(int(x[2 * pair])), oracle.u01(int(x[2 * pair + 1])))
            assert abs(noise[t] - g[h % 2]) < 1e-9, (h, t)
    n = np.concatenate(draws)
    assert stats.kstest(n, "norm").pvalue > 1e-4
    assert abs(np.corrcoef(draws[0], draws[1])[0, 1]) < 0.02
    # another stream draws other numbers
    other = source_of(arch, f0, np.eye(H1)[0], seed=seed, stream=stream + 1)
    assert np.abs(np.arctanh(other) / (A / 3.0) - draws[0]).mean() > 0.5


def test_constant_f0_sinusoids_closed_form():
    """Voiced constant f0, no noise: sinusoid h is A sin(2 pi ((h+1) f0 (t+1)/sr + phi_h)),
    phi_0 = 0, phi_h the first draw of counter (0, h, 1, 0)."""
    arch = dict(TINY_SRC, noise_std=0.0)
    A, sr = arch["sine_amp"], arch["sample_rate"]
    H1 = arch["n_harmonics"] + 1
    F = 30
    f0v = 217.3
    t = np.arange(F * SPF, dtype=np.float64)
    seed, stream = 9, 0
    for h in range(H1):
        merge = np.zeros(H1)
        merge[h] = 1.0
        src = source_of(arch, np.full(F, f0v), merge, seed=seed, stream=stream)
        phi = 0.0 if h == 0 else oracle.u01(int(np_philox((0, h, 1, 0), (seed, stream))[0]))
        want = np.tanh(A * np.sin(2 * np.pi * ((h + 1) * f0v * (t + 1) / sr + phi)))
        assert np.abs(src - want).max() < 1e-9, h


def test_piecewise_f0_phase_is_a_running_sum():
    """Per-frame f0 (voiced and unvoiced frames): the phase of sample t is the
    running sum of the per-sample increments (h+1) f0 / sr up to t, summed
    here directly with numpy; unvoiced frames carry no sinusoid but still
    advance the phase by their (sub-threshold) f0, and hold the same noise
    as an all-unvoiced contour (the draws depend on the sample, not on f0)."""
    arch = dict(TINY_SRC, noise_std=0.0)
    A, sr, thr = arch["sine_amp"], arch["sample_rate"], arch["voiced_threshold"]
    H1 = arch["n_harmonics"] + 1
    rng = np.random.default_rng(3)
    F = 50
    f0 = rng.uniform(70, 450, F)
    f0[rng.random(F) < 0.3] = 0.0
    f0[7] = 5.0                                          # below the voicing threshold, non-zero
    seed, stream = 1, 4
    per_sample = np.repeat(f0, SPF)
    voiced = per_sample > thr
    for h in range(H1):
        merge = np.zeros(H1)
        merge[h] = 1.0
        src = source_of(arch, f0, merge, seed=seed, stream=stream)
        phi = 0.0 if h == 0 else oracle.u01(int(np_philox((0, h, 1, 0), (seed, stream))[0]))
        phase = phi + np.cumsum((h + 1) * per_sample / sr)
        noise_only = source_of(arch, np.zeros(F), merge, seed=seed, stream=stream)
        want = np.where(voiced, np.tanh(A * np.sin(2 * np.pi * phase)), noise_only)
        assert np.abs(src - want).max() < 1e-9, h


def test_merge_weights_and_bias():
    arch = TINY_SRC
    H1 = arch["n_harmonics"] + 1
    f0 = synth.make_f0(arch, 1, 30)[0]
    parts = [np.arctanh(source_of(arch, f0, np.eye(H1)[h])) for h in range(H1)]
    w = np.array([0.7, -1.3, 0.2])[:H1]
    src = source_of(arch, f0, w, merge_b=0.05)
    want = np.tanh(0.05 + sum(w[h] * parts[h] for h in range(H1)))
    assert np.abs(src - want).max() < 1e-12


def planted_nsf(arch, seed=0):
    blob = synth.make_weights(arch, seed)
    return blob, synth.split_weights(arch, blob)


def test_source_enters_after_the_last_upsampling():
    """Zero down-conv weights and bias c: the decoder equals the one without a
    source whose last ConvTranspose1d bias is raised by c."""
    arch = synth.TINY_NSF_ARCH
    plain_arch = synth.TINY_ARCH
    blob, W = planted_nsf(arch)
    L = len(arch["up_rate"]) - 1
    c = np.linspace(-0.2, 0.3, arch["channels"][-1]).astype(np.float32)
    W["src.down.W"][:] = 0.0
    W["src.down.b"][:] = c
    ids = synth.make_tokens(arch, 1, 12)[0]
    f0 = synth.make_f0(arch, 1, 12)[0]
    pcm = oracle.decode(arch, "f32", blob, ids, f0=f0, seed=3)
    plain = blob[:synth.blob_floats(plain_arch)].copy()
    Wp = synth.split_weights(plain_arch, plain)
    Wp[f"s{L}.up.b"][:] = Wp[f"s{L}.up.b"] + c.astype(np.float64)
    want = oracle.decode(plain_arch, "f32", plain, ids)
    # (the raised bias is stored in float32: its rounding is the only difference)
    assert np.abs(pcm - want).max() <= 1e-6 * np.abs(want).max()
    assert np.abs(pcm - oracle.decode(plain_arch, "f32", blob[:plain.size], ids)).max() > 1e-3


def test_down_conv_reads_the_frame_samples():
    """A one-hot down-conv weight W[c0][0][j0] = 1 adds src[4 tau + j0] to channel
    c0 of the last stage's ConvTranspose1d output at frame tau, and nothing else."""
    arch = synth.TINY_NSF_ARCH
    blob, W = planted_nsf(arch, 1)
    L = len(arch["up_rate"]) - 1
    W["src.down.W"][:] = 0.0
    W["src.down.b"][:] = 0.0
    c0, j0 = 5, 2
    W["src.down.W"][c0, 0, j0] = 1.0
    ids = synth.make_tokens(arch, 1, 10, seed=4)[0]
    f0 = synth.make_f0(arch, 1, 10, seed=4)[0]
    _, y = oracle.decode(arch, "f32", blob, ids, tap=f"s{L}.y", f0=f0, seed=7)
    _, src = oracle.decode(arch, "f32", blob, ids, tap="src", f0=f0, seed=7)
    W["src.down.W"][c0, 0, j0] = 0.0
    _, y0 = oracle.decode(arch, "f32", blob, ids, tap=f"s{L}.y", f0=f0, seed=7)
    d = y - y0
    assert np.abs(np.delete(d, c0, axis=1)).max() == 0.0
    assert np.abs(d[:, c0] - src[:, j0]).max() < 1e-12
    assert src.shape == (y.shape[0], arch["hop"])


def test_real_source_statistics():
    """The excitation of the real architecture on a synthetic contour: bounded
    by tanh, voiced frames carry the sinusoids (larger RMS than unvoiced)."""
    arch = synth.REAL_NSF_ARCH
    H1 = arch["n_harmonics"] + 1
    f0 = synth.make_f0(arch, 1, 25)[0]
    src = source_of(arch, f0, np.ones(H1) / H1, seed=0, stream=0)
    S = arch["hop"] * math.prod(arch["up_rate"])
    v = np.repeat(f0 > arch["voiced_threshold"], S)
    assert src.size == f0.size * S and np.abs(src).max() < 1.0
    assert v.any() and (~v).any()
    assert np.sqrt(np.mean(src[v] ** 2)) > 2.0 * np.sqrt(np.mean(src[~v] ** 2))
