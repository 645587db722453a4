"""ctypes driver of the plain C oracle (oracle.c).

TEST INFRASTRUCTURE ONLY: the tests, the smoke check and the benchmark's CPU
baseline leg may import this package; the product path never does.  It shares
no code with the GPU library.  `build()` compiles liboracle.so with gcc.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.c")
_SRCS = [_SRC, os.path.join(_HERE, "flow.c")]
_LIB = os.path.join(_HERE, "liboracle.so")
_lib = None


def build() -> str:
    """Compile the oracle (plain C, fp64, OpenMP over output frames)."""
    tmp = _LIB + ".tmp"
    subprocess.run(["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-Wall", "-std=gnu11",
                    "-o", tmp, *_SRCS, "-lm"], check=True)
    os.replace(tmp, _LIB)
    return _LIB


def build_sanitized(out: str) -> str:
    """The same sources with AddressSanitizer and UndefinedBehaviorSanitizer
    (host code, gcc; single-threaded, any sanitizer report aborts the
    process).  Load it by setting DC_ORACLE_LIB to `out` in a process started
    with the sanitizer runtime preloaded."""
    subprocess.run(["gcc", "-O1", "-g", "-fno-omit-frame-pointer", "-fsanitize=address,undefined",
                    "-fno-sanitize-recover=all", "-fPIC", "-shared", "-Wall", "-Wno-unknown-pragmas",
                    "-std=gnu11", "-o", out, *_SRCS, "-lm"], check=True)
    return out


class _Arch(ctypes.Structure):
    _fields_ = [
        ("vocab", ctypes.c_int), ("embed", ctypes.c_int), ("frames_per_token", ctypes.c_int),
        ("n_pre", ctypes.c_int), ("pre_kernel", ctypes.c_int),
        ("n_stages", ctypes.c_int), ("up_rate", ctypes.c_int * 8), ("channels", ctypes.c_int * 9),
        ("n_rb", ctypes.c_int), ("rb_kernel", ctypes.c_int * 8),
        ("n_dil", ctypes.c_int), ("dil", ctypes.c_int * 8),
        ("head_kernel", ctypes.c_int), ("n_fft", ctypes.c_int), ("hop", ctypes.c_int),
        ("slope", ctypes.c_double),
        ("n_harmonics", ctypes.c_int),
        ("sine_amp", ctypes.c_double), ("noise_std", ctypes.c_double),
        ("voiced_threshold", ctypes.c_double), ("sample_rate", ctypes.c_double),
    ]


def _load():
    global _lib
    if _lib is None:
        path = os.environ.get("DC_ORACLE_LIB")   # a sanitized build (tests)
        if path is None:
            path = _LIB
            if not os.path.exists(_LIB) or os.path.getmtime(_LIB) < max(os.path.getmtime(f) for f in _SRCS):
                build()
        lib = ctypes.CDLL(path)
        D = ctypes.POINTER(ctypes.c_double)
        F = ctypes.POINTER(ctypes.c_float)
        I = ctypes.POINTER(ctypes.c_int32)
        lib.oc_cconv.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_long,
                                 D, D, D, D]
        lib.oc_convt.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_long, D, D, D, D]
        lib.oc_irfft.argtypes = [ctypes.c_int, D, D, D]
        lib.oc_istft.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_long, D, D, D]
        lib.oc_hann.argtypes = [ctypes.c_int, ctypes.c_int]
        lib.oc_hann.restype = ctypes.c_double
        lib.oc_ola_norm.argtypes = [ctypes.c_int, ctypes.c_int]
        lib.oc_ola_norm.restype = ctypes.c_double
        lib.oc_round_bf16.argtypes = [ctypes.c_float]
        lib.oc_round_bf16.restype = ctypes.c_float
        lib.oc_num_threads.restype = ctypes.c_int
        lib.oc_blob_floats.argtypes = [ctypes.POINTER(_Arch)]
        lib.oc_blob_floats.restype = ctypes.c_long
        lib.oc_samples_per_token.argtypes = [ctypes.POINTER(_Arch)]
        lib.oc_samples_per_token.restype = ctypes.c_long
        lib.oc_decode.argtypes = [ctypes.POINTER(_Arch), ctypes.c_int, F, ctypes.c_long, I, ctypes.c_long,
                                  D, ctypes.c_uint64, ctypes.c_uint64, D, ctypes.c_char_p, D]
        lib.oc_decode.restype = ctypes.c_int
        U64 = ctypes.POINTER(ctypes.c_uint64)
        lib.oc_philox4x64.argtypes = [U64, U64, U64]
        lib.oc_u01.argtypes = [ctypes.c_uint64]
        lib.oc_u01.restype = ctypes.c_double
        lib.oc_box_muller.argtypes = [ctypes.c_double, ctypes.c_double, D, D]
        lib.oc_source.argtypes = [ctypes.POINTER(_Arch), D, ctypes.c_long, ctypes.c_uint64, ctypes.c_uint64,
                                  D, ctypes.c_double, D]
        FP = ctypes.POINTER(_FlowArch)
        V = ctypes.c_void_p
        lib.ocf_blob_floats.argtypes = [FP]
        lib.ocf_blob_floats.restype = ctypes.c_long
        lib.ocf_open.argtypes = [FP, ctypes.c_int, F, ctypes.c_long, ctypes.c_uint64, ctypes.c_uint64]
        lib.ocf_open.restype = V
        lib.ocf_close.argtypes = [V]
        lib.ocf_prompt.argtypes = [V, ctypes.c_int, D, D, D, D]
        lib.ocf_prompt.restype = ctypes.c_int
        lib.ocf_chunk.argtypes = [V, ctypes.c_int, D, D]
        lib.ocf_chunk.restype = ctypes.c_int
        lib.ocf_carry.argtypes = [V, ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_int, D]
        lib.ocf_carry.restype = ctypes.c_int
        lib.ocf_position.argtypes = [V]
        lib.ocf_position.restype = ctypes.c_int64
        lib.ocf_get_times.argtypes = [V, D]
        lib.ocf_get_mods.argtypes = [V, ctypes.c_int, ctypes.c_int, D]
        lib.ocf_times.argtypes = [ctypes.c_int, D]
        lib.ocf_time_embedding.argtypes = [ctypes.c_int, ctypes.c_double, D]
        lib.ocf_gelu.argtypes = [ctypes.c_double]
        lib.ocf_gelu.restype = ctypes.c_double
        lib.ocf_lnmod.argtypes = [ctypes.c_int, D, D, D, D]
        lib.ocf_attention.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_int, D, D, D, ctypes.c_int, D]
        lib.ocf_noise.argtypes = [ctypes.c_int, ctypes.c_double, ctypes.c_uint64, ctypes.c_uint64,
                                  ctypes.c_int64, ctypes.c_int, D]
        _lib = lib
    return _lib


class _FlowArch(ctypes.Structure):
    _fields_ = [
        ("n_mel", ctypes.c_int), ("dim", ctypes.c_int), ("heads", ctypes.c_int), ("depth", ctypes.c_int),
        ("mlp", ctypes.c_int), ("t_dim", ctypes.c_int), ("n_steps", ctypes.c_int),
        ("f_prompt", ctypes.c_int), ("f_retained", ctypes.c_int), ("f_chunk", ctypes.c_int),
        ("f_call", ctypes.c_int), ("cfg_rate", ctypes.c_double), ("temperature", ctypes.c_double),
    ]


def _p(a: np.ndarray, ct):
    return a.ctypes.data_as(ctypes.POINTER(ct))


def _f64(a) -> np.ndarray:
    return np.ascontiguousarray(a, dtype=np.float64)


def arch_struct(arch: dict) -> _Arch:
    s = _Arch()
    s.vocab, s.embed, s.frames_per_token = arch["vocab"], arch["embed"], arch["frames_per_token"]
    s.n_pre, s.pre_kernel = arch["n_pre"], arch["pre_kernel"]
    s.n_stages = len(arch["up_rate"])
    for i, u in enumerate(arch["up_rate"]):
        s.up_rate[i] = u
    for i, c in enumerate(arch["channels"]):
        s.channels[i] = c
    s.n_rb = len(arch["rb_kernel"])
    for i, k in enumerate(arch["rb_kernel"]):
        s.rb_kernel[i] = k
    s.n_dil = len(arch["dil"])
    for i, d in enumerate(arch["dil"]):
        s.dil[i] = d
    s.head_kernel, s.n_fft, s.hop = arch["head_kernel"], arch["n_fft"], arch["hop"]
    s.slope = arch["lrelu_slope"]
    s.n_harmonics = arch.get("n_harmonics", 0)
    s.sine_amp = arch.get("sine_amp", 0.0)
    s.noise_std = arch.get("noise_std", 0.0)
    s.voiced_threshold = arch.get("voiced_threshold", 0.0)
    s.sample_rate = arch.get("sample_rate", 1.0)
    return s


# ---------------------------------------------------------------- single ops

def cconv(W, b, v, d: int = 1) -> np.ndarray:
    """Causal dilated conv: W [Co][Ci][k], b [Co], v [T][Ci] -> [T][Co]."""
    W, b, v = _f64(W), _f64(b), _f64(v)
    co, ci, k = W.shape
    T = v.shape[0]
    out = np.empty((T, co), dtype=np.float64)
    _load().oc_cconv(ci, co, k, d, T, _p(W, ctypes.c_double), _p(b, ctypes.c_double),
                     _p(v, ctypes.c_double), _p(out, ctypes.c_double))
    return out


def convt(W, b, v) -> np.ndarray:
    """Causal transposed conv, kernel 2u stride u: W [Ci][Co][2u], v [F][Ci] -> [F*u][Co]."""
    W, b, v = _f64(W), _f64(b), _f64(v)
    ci, co, k2 = W.shape
    u = k2 // 2
    F = v.shape[0]
    out = np.empty((F * u, co), dtype=np.float64)
    _load().oc_convt(ci, co, u, F, _p(W, ctypes.c_double), _p(b, ctypes.c_double),
                     _p(v, ctypes.c_double), _p(out, ctypes.c_double))
    return out


def irfft(re, im) -> np.ndarray:
    re, im = _f64(re), _f64(im)
    N = 2 * (re.size - 1)
    out = np.empty(N, dtype=np.float64)
    _load().oc_irfft(N, _p(re, ctypes.c_double), _p(im, ctypes.c_double), _p(out, ctypes.c_double))
    return out


def istft(logmag, phase, n_fft: int = 16, hop: int = 4) -> np.ndarray:
    """[M][n_fft/2+1] log-magnitude and phase -> hop*M samples."""
    lm, ph = _f64(logmag), _f64(phase)
    M = lm.shape[0]
    out = np.empty(M * hop, dtype=np.float64)
    _load().oc_istft(n_fft, hop, M, _p(lm, ctypes.c_double), _p(ph, ctypes.c_double),
                     _p(out, ctypes.c_double))
    return out


def hann(N: int) -> np.ndarray:
    lib = _load()
    return np.array([lib.oc_hann(N, n) for n in range(N)])


def ola_norm(N: int, hop: int) -> float:
    return _load().oc_ola_norm(N, hop)


def round_bf16(x) -> np.ndarray:
    lib = _load()
    x = np.asarray(x, dtype=np.float32)
    return np.array([lib.oc_round_bf16(float(v)) for v in x.ravel()], dtype=np.float32).reshape(x.shape)


def philox4x64(ctr, key) -> np.ndarray:
    """Philox4x64-10 block of counter ctr (4 x uint64) under key (2 x uint64)."""
    c = np.ascontiguousarray(ctr, dtype=np.uint64)
    k = np.ascontiguousarray(key, dtype=np.uint64)
    out = np.empty(4, dtype=np.uint64)
    _load().oc_philox4x64(_p(c, ctypes.c_uint64), _p(k, ctypes.c_uint64), _p(out, ctypes.c_uint64))
    return out


def u01(x: int) -> float:
    return _load().oc_u01(int(x))


def box_muller(u0: float, u1: float):
    g0, g1 = ctypes.c_double(), ctypes.c_double()
    _load().oc_box_muller(u0, u1, ctypes.byref(g0), ctypes.byref(g1))
    return g0.value, g1.value


def source(arch: dict, f0, seed: int, stream: int, merge_w, merge_b: float) -> np.ndarray:
    """Harmonic-plus-noise excitation of one stream: f0 [F] (Hz, pre-stack
    frame clock) -> F * prod(up_rate) * hop samples."""
    s = arch_struct(arch)
    f0 = _f64(f0).ravel()
    mw = _f64(merge_w).ravel()
    S = arch["hop"]
    for u in arch["up_rate"]:
        S *= u
    out = np.empty(f0.size * S, dtype=np.float64)
    _load().oc_source(ctypes.byref(s), _p(f0, ctypes.c_double), f0.size, seed, stream,
                      _p(mw, ctypes.c_double), float(merge_b), _p(out, ctypes.c_double))
    return out


def num_threads() -> int:
    return _load().oc_num_threads()


def samples_per_token(arch: dict) -> int:
    s = arch_struct(arch)
    return int(_load().oc_samples_per_token(ctypes.byref(s)))


# ---------------------------------------------------------------- the decoder

def decode(arch: dict, dtype: str, blob: np.ndarray, ids, tap: str | None = None, f0=None,
           seed: int = 0, stream: int = 0):
    """Offline decode of one stream from the zero state.

    Returns the fp64 PCM (len(ids) * samples_per_token samples), or
    (pcm, tap_values) when `tap` names an intermediate.  dtype "bf16" rounds
    every parameter to bfloat16 first.  An architecture with a harmonic
    source takes f0 (len(ids) * frames_per_token values, Hz) and the
    generator's (seed, stream) key.
    """
    lib = _load()
    s = arch_struct(arch)
    blob = np.ascontiguousarray(blob, dtype=np.float32)
    ids = np.ascontiguousarray(ids, dtype=np.int32).ravel()
    T = ids.size
    f0a = None
    if arch.get("n_harmonics", 0) > 0:
        f0a = _f64(f0).ravel()
        if f0a.size != T * arch["frames_per_token"]:
            raise ValueError("f0 needs len(ids) * frames_per_token values")
    spt = int(lib.oc_samples_per_token(ctypes.byref(s)))
    pcm = np.empty(T * spt, dtype=np.float64)
    tap_buf = None
    if tap is not None:
        frames, ch = _tap_shape(arch, tap, T)
        tap_buf = np.empty((frames, ch), dtype=np.float64)
    rc = lib.oc_decode(ctypes.byref(s), 1 if dtype == "bf16" else 0, _p(blob, ctypes.c_float), blob.size,
                       _p(ids, ctypes.c_int32), T,
                       _p(f0a, ctypes.c_double) if f0a is not None else None, seed, stream,
                       _p(pcm, ctypes.c_double),
                       tap.encode() if tap else None,
                       _p(tap_buf, ctypes.c_double) if tap_buf is not None else None)
    if rc != 0:
        raise ValueError(f"oracle decode failed (rc={rc})")
    return pcm if tap is None else (pcm, tap_buf)


def _tap_shape(arch: dict, tap: str, T: int):
    F = T * arch["frames_per_token"]
    if tap == "embed" or tap.startswith("pre"):
        return F, arch["channels"][0]
    if tap in ("head", "src"):
        for u in arch["up_rate"]:
            F *= u
        return F, 2 * (arch["n_fft"] // 2 + 1) if tap == "head" else arch["hop"]
    s = int(tap[1:tap.index(".")])
    for u in arch["up_rate"][:s + 1]:
        F *= u
    return F, arch["channels"][s + 1]


# ------------------------------------------------------------ the flow decoder

def flow_arch_struct(arch: dict) -> _FlowArch:
    s = _FlowArch()
    for name, _ in _FlowArch._fields_:
        setattr(s, name, arch[name])
    return s


def flow_times(n: int) -> np.ndarray:
    t = np.empty(n + 1, dtype=np.float64)
    _load().ocf_times(n, _p(t, ctypes.c_double))
    return t


def flow_time_embedding(t_dim: int, t: float) -> np.ndarray:
    e = np.empty(t_dim, dtype=np.float64)
    _load().ocf_time_embedding(t_dim, float(t), _p(e, ctypes.c_double))
    return e


def gelu(v: float) -> float:
    return _load().ocf_gelu(float(v))


def lnmod(h, shift, scale) -> np.ndarray:
    h, shift, scale = _f64(h).ravel(), _f64(shift).ravel(), _f64(scale).ravel()
    out = np.empty_like(h)
    _load().ocf_lnmod(h.size, _p(h, ctypes.c_double), _p(shift, ctypes.c_double), _p(scale, ctypes.c_double),
                      _p(out, ctypes.c_double))
    return out


def attention(q, k, v) -> np.ndarray:
    """One head: q [nq][hd], k, v [nk][hd] -> [nq][hd]."""
    q, k, v = _f64(q), _f64(k), _f64(v)
    out = np.empty_like(q)
    _load().ocf_attention(q.shape[0], k.shape[0], q.shape[1], _p(q, ctypes.c_double), _p(k, ctypes.c_double),
                          _p(v, ctypes.c_double), q.shape[1], _p(out, ctypes.c_double))
    return out


def flow_noise(n_mel: int, temperature: float, seed: int, key: int, tau0: int, frames: int) -> np.ndarray:
    out = np.empty((frames, n_mel), dtype=np.float64)
    _load().ocf_noise(n_mel, temperature, seed, key, tau0, frames, _p(out, ctypes.c_double))
    return out


class FlowStream:
    """One stream of the flow decoder in fp64: prompt(), then chunk() calls.

    dtype "bf16" rounds the per-step Linear weights to bfloat16 first.
    """

    def __init__(self, arch: dict, dtype: str, blob: np.ndarray, seed: int = 0, key: int = 0):
        self.arch = dict(arch)
        self._a = flow_arch_struct(arch)
        self._blob = np.ascontiguousarray(blob, dtype=np.float32)
        self._lib = _load()
        self._h = self._lib.ocf_open(ctypes.byref(self._a), 1 if dtype == "bf16" else 0,
                                     _p(self._blob, ctypes.c_float), self._blob.size, seed, key)
        if not self._h:
            raise ValueError("bad flow architecture or blob size")

    def close(self):
        if self._h:
            self._lib.ocf_close(self._h)
            self._h = None

    def __del__(self):
        self.close()

    def prompt(self, mu, cond, spk) -> np.ndarray:
        mu, cond, spk = _f64(mu), _f64(cond), _f64(spk).ravel()
        P = mu.shape[0]
        mel = np.empty((P, self.arch["n_mel"]), dtype=np.float64)
        if self._lib.ocf_prompt(self._h, P, _p(mu, ctypes.c_double), _p(cond, ctypes.c_double),
                                _p(spk, ctypes.c_double), _p(mel, ctypes.c_double)) != 0:
            raise ValueError("prompt length out of range")
        return mel

    def chunk(self, mu) -> np.ndarray:
        mu = _f64(mu)
        n = mu.shape[0]
        mel = np.empty((n, self.arch["n_mel"]), dtype=np.float64)
        self.extent = self._lib.ocf_chunk(self._h, n, _p(mu, ctypes.c_double), _p(mel, ctypes.c_double))
        if self.extent < 0:
            raise ValueError("chunk before a prompt, or frame count out of range")
        return mel

    def carry(self, step: int, layer: int, branch: int, kv: int) -> np.ndarray:
        n = self._lib.ocf_carry(self._h, step, layer, branch, kv, None)
        out = np.empty((n, self.arch["dim"]), dtype=np.float64)
        self._lib.ocf_carry(self._h, step, layer, branch, kv, _p(out, ctypes.c_double))
        return out

    @property
    def position(self) -> int:
        return int(self._lib.ocf_position(self._h))

    def times(self) -> np.ndarray:
        t = np.empty(self.arch["n_steps"] + 1, dtype=np.float64)
        self._lib.ocf_get_times(self._h, _p(t, ctypes.c_double))
        return t

    def mods(self, step: int, layer: int) -> np.ndarray:
        """[6][dim] modulation of block `layer` at solver step `step` ([2][dim] for layer == depth)."""
        D = self.arch["dim"]
        k = 6 if layer < self.arch["depth"] else 2
        out = np.empty(k * D, dtype=np.float64)
        self._lib.ocf_get_mods(self._h, step, layer, _p(out, ctypes.c_double))
        return out.reshape(k, D)
