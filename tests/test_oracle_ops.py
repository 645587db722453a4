"""Pins of the oracle's single operations against library routines, closed
forms and identities that do not share its code (CPU only)."""
import math

import numpy as np
import pytest
import scipy.signal
import torch
import torch.nn.functional as F

import oracle


def _rng(seed):
    return np.random.default_rng(seed)


# ------------------------------------------------------------ causal conv

@pytest.mark.parametrize("ci,co,k,d,T", [(3, 5, 3, 1, 17), (8, 4, 7, 3, 40), (6, 6, 11, 5, 90), (4, 18, 7, 1, 9)])
def test_cconv_matches_torch_conv1d_left_padded(ci, co, k, d, T):
    r = _rng(ci * 100 + k)
    W, b, v = r.standard_normal((co, ci, k)), r.standard_normal(co), r.standard_normal((T, ci))
    ref = F.conv1d(F.pad(torch.tensor(v.T[None]), ((k - 1) * d, 0)), torch.tensor(W), torch.tensor(b),
                   dilation=d)[0].numpy().T
    np.testing.assert_allclose(oracle.cconv(W, b, v, d), ref, rtol=0, atol=1e-12)


def test_cconv_identity_and_delay():
    """W = delta at the last tap is the identity; at the first tap it delays by (k-1)d."""
    r = _rng(1)
    C, k, d, T = 4, 5, 3, 30
    v, b = r.standard_normal((T, C)), r.standard_normal(C)
    W = np.zeros((C, C, k))
    W[np.arange(C), np.arange(C), k - 1] = 1.0
    np.testing.assert_array_equal(oracle.cconv(W, b, v, d), v + b)
    W = np.zeros((C, C, k))
    W[np.arange(C), np.arange(C), 0] = 1.0
    out = oracle.cconv(W, np.zeros(C), v, d)
    lag = (k - 1) * d
    np.testing.assert_array_equal(out[lag:], v[:T - lag])
    np.testing.assert_array_equal(out[:lag], 0.0)


def test_cconv_channel_mixing_orientation():
    """out[o] takes input channel i through W[o][i]: a single 1 at W[1][2] copies channel 2 to 1."""
    T, k = 6, 3
    v = np.arange(T * 3, dtype=float).reshape(T, 3)
    W = np.zeros((2, 3, k))
    W[1, 2, k - 1] = 1.0
    out = oracle.cconv(W, np.zeros(2), v)
    np.testing.assert_array_equal(out[:, 1], v[:, 2])
    np.testing.assert_array_equal(out[:, 0], 0.0)


# ------------------------------------------------------ transposed conv

@pytest.mark.parametrize("ci,co,u,Fr", [(3, 2, 2, 5), (8, 4, 8, 7), (6, 5, 5, 4), (4, 4, 3, 9)])
def test_convt_matches_torch_conv_transpose1d_truncated(ci, co, u, Fr):
    r = _rng(ci + 10 * u)
    W, b, v = r.standard_normal((ci, co, 2 * u)), r.standard_normal(co), r.standard_normal((Fr, ci))
    ref = F.conv_transpose1d(torch.tensor(v.T[None]), torch.tensor(W), torch.tensor(b),
                             stride=u)[0].numpy().T[:Fr * u]
    np.testing.assert_allclose(oracle.convt(W, b, v), ref, rtol=0, atol=1e-12)


@pytest.mark.parametrize("u", [2, 3, 5, 8])
def test_convt_equals_zero_stuffed_causal_conv(u):
    """ConvTranspose1d(k=2u, stride u) == causal conv of the zero-stuffed input
    with W'[o][i][j] = W[i][o][2u-1-j]."""
    r = _rng(u)
    ci, co, Fr = 5, 3, 11
    W, b, v = r.standard_normal((ci, co, 2 * u)), r.standard_normal(co), r.standard_normal((Fr, ci))
    stuffed = np.zeros((Fr * u, ci))
    stuffed[::u] = v
    Wp = np.flip(W, axis=2).transpose(1, 0, 2)
    np.testing.assert_allclose(oracle.convt(W, b, v), oracle.cconv(Wp, b, stuffed), rtol=0, atol=1e-12)


# ----------------------------------------------------------- iDFT / iSTFT

def test_irfft_matches_numpy():
    r = _rng(3)
    for N in (8, 16, 32):
        X = r.standard_normal(N // 2 + 1) + 1j * r.standard_normal(N // 2 + 1)
        np.testing.assert_allclose(oracle.irfft(X.real, X.imag), np.fft.irfft(X, N), rtol=0, atol=1e-13)


def test_hann_is_periodic_hann():
    np.testing.assert_allclose(oracle.hann(16), scipy.signal.get_window("hann", 16, fftbins=True),
                               rtol=0, atol=1e-15)


def test_cola_constants():
    """Periodic Hann at hop N/4: sum_m w = 2 and sum_m w^2 = 1.5 at every n."""
    w = scipy.signal.get_window("hann", 16, fftbins=True)
    for n in range(4):
        assert math.isclose(sum(w[n + 4 * m] for m in range(4)), 2.0, abs_tol=1e-15)
    assert math.isclose(oracle.ola_norm(16, 4), 1.5, abs_tol=1e-15)


def test_istft_inverts_stft():
    """iSTFT(STFT(x)) == x for every fully overlapped sample (t >= N - hop)."""
    N, hop, M = 16, 4, 60
    r = _rng(7)
    x = r.standard_normal(hop * (M - 1) + N)
    w = scipy.signal.get_window("hann", N, fftbins=True)
    X = np.stack([np.fft.rfft(w * x[hop * m: hop * m + N]) for m in range(M)])
    rec = oracle.istft(np.log(np.abs(X)), np.angle(X), N, hop)
    np.testing.assert_allclose(rec[N - hop:], x[N - hop: hop * M], rtol=0, atol=1e-12)


def test_istft_pulse_train_closed_form():
    """log|X| = 0 and phase = -pi*kk give X_kk = (-1)^kk, an impulse at n = 8 in
    every frame, w[8] = 1, hence 1/1.5 at t = 4m + 8 and 0 elsewhere."""
    M = 20
    lm = np.zeros((M, 9))
    ph = np.tile(-np.pi * np.arange(9), (M, 1))
    pcm = oracle.istft(lm, ph)
    t = np.arange(4 * M)
    ref = np.where((t % 4 == 0) & (t >= 8), 2.0 / 3.0, 0.0)
    np.testing.assert_allclose(pcm, ref, rtol=0, atol=1e-14)


def test_istft_zero_spectrum_phase_gives_silence():
    """log|X| = 0, phase = 0: every frame is an impulse at n = 0 where w[0] = 0."""
    pcm = oracle.istft(np.zeros((10, 9)), np.zeros((10, 9)))
    np.testing.assert_allclose(pcm, 0.0, atol=1e-15)


# ------------------------------------------------------------ bf16 rounding

def test_round_bf16_matches_torch():
    r = _rng(11)
    x = np.concatenate([r.standard_normal(2000).astype(np.float32) * 10.0 ** r.integers(-6, 6, 2000),
                        np.array([1.0 + 2.0 ** -8, 1.0 + 3 * 2.0 ** -8, -(1.0 + 2.0 ** -8), 0.0, -0.0,
                                  3.0e38, 1e-40], dtype=np.float32)])
    ref = torch.tensor(x).to(torch.bfloat16).to(torch.float32).numpy()
    np.testing.assert_array_equal(oracle.round_bf16(x), ref)
