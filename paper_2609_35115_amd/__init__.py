"""MI355X streaming Token2Wav decode step: Python binding of libdc.so.

The functions below carry the C-ABI names of include/dc.h and only marshal
arguments (torch tensors or numpy arrays to pointers); every step of the
decode runs in the gfx950 kernels of libdc.so.  Importing this package never
falls back to anything else: if libdc.so is missing, `lib()` raises.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

from . import synth  # noqa: F401  (workload shapes and seeded inputs)

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libdc.so")

DC_ABI_VERSION = 3
DC_OK, DC_EINVAL, DC_ERANGE, DC_ENOMEM, DC_EDEVICE, DC_ESTATE, DC_EVERSION = 0, -1, -2, -3, -4, -5, -6
DC_F32, DC_BF16 = 0, 1
DC_HOST_PTRS, DC_NO_GRAPH, DC_NO_FUSE, DC_FLUSH_CATALOG, DC_NO_RING = 1, 2, 4, 8, 16
STATUS_NAMES = {0: "DC_OK", -1: "DC_EINVAL", -2: "DC_ERANGE", -3: "DC_ENOMEM", -4: "DC_EDEVICE",
                -5: "DC_ESTATE", -6: "DC_EVERSION"}


class DcError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"{STATUS_NAMES.get(status, status)}: {msg}")
        self.status = status


class DcCfg(ctypes.Structure):
    _fields_ = [
        ("abi_version", ctypes.c_int32),
        ("vocab", ctypes.c_int32), ("embed", ctypes.c_int32),
        ("frames_per_token", ctypes.c_int32),
        ("n_pre", ctypes.c_int32), ("pre_kernel", ctypes.c_int32),
        ("n_stages", ctypes.c_int32),
        ("up_rate", ctypes.c_int32 * 4),
        ("channels", ctypes.c_int32 * 5),
        ("n_rb", ctypes.c_int32), ("rb_kernel", ctypes.c_int32 * 4),
        ("n_dil", ctypes.c_int32), ("dil", ctypes.c_int32 * 4),
        ("head_kernel", ctypes.c_int32), ("n_fft", ctypes.c_int32), ("hop", ctypes.c_int32),
        ("lrelu_slope", ctypes.c_float),
        ("dtype", ctypes.c_int32),
        ("batch", ctypes.c_int32),
        ("chunk_tokens", ctypes.c_int32),
        ("max_tokens", ctypes.c_int32),
        ("flags", ctypes.c_uint32),
        ("tile_variant", ctypes.c_int32),
        ("n_harmonics", ctypes.c_int32),
        ("sine_amp", ctypes.c_float), ("noise_std", ctypes.c_float),
        ("voiced_threshold", ctypes.c_float), ("sample_rate", ctypes.c_float),
        ("rng_seed", ctypes.c_uint64),
        ("hip_stream", ctypes.c_void_p),
    ]


class DcStats(ctypes.Structure):
    _fields_ = [
        ("calls", ctypes.c_int64), ("replays", ctypes.c_int64), ("direct_shape", ctypes.c_int64),
        ("direct_nograph", ctypes.c_int64), ("staged_tokens", ctypes.c_int64),
        ("staged_audio", ctypes.c_int64), ("rejected", ctypes.c_int64), ("clock_tokens", ctypes.c_int64),
        ("arena_bytes", ctypes.c_int64), ("weight_bytes", ctypes.c_int64), ("carry_bytes", ctypes.c_int64),
        ("ring_bytes", ctypes.c_int64), ("kernels_per_step", ctypes.c_int32), ("graph_nodes", ctypes.c_int32),
        ("capture_ms", ctypes.c_double), ("replays_flush", ctypes.c_int64), ("graph_classes", ctypes.c_int32),
        ("reserved", ctypes.c_int32), ("staged_f0", ctypes.c_int64), ("direct_static", ctypes.c_int64),
    ]

    def as_dict(self) -> dict:
        return {name: getattr(self, name) for name, _ in self._fields_}


class DcLayerInfo(ctypes.Structure):
    _fields_ = [("name", ctypes.c_char * 48), ("kernel", ctypes.c_char * 80),
                ("rows", ctypes.c_int64), ("cols", ctypes.c_int64), ("depth", ctypes.c_int64),
                ("flops", ctypes.c_double), ("bytes", ctypes.c_double)]


# Every symbol include/dc.h declares, with its ctypes signature.
_P = ctypes.c_void_p
SIGNATURES = {
    "dc_init": ([_P, ctypes.c_size_t, ctypes.POINTER(DcCfg), ctypes.POINTER(_P)], ctypes.c_int),
    "dc_decode_chunk": ([_P, _P, ctypes.c_int32, _P], ctypes.c_int),
    "dc_decode_chunk_f0": ([_P, _P, _P, ctypes.c_int32, _P], ctypes.c_int),
    "dc_decode_chunk_f0_static": ([_P, _P, _P, ctypes.c_int32, _P], ctypes.c_int),
    "dc_reset": ([_P], ctypes.c_int),
    "dc_reset_stream": ([_P, ctypes.c_int32], ctypes.c_int),
    "dc_sync": ([_P], ctypes.c_int),
    "dc_samples_per_token": ([ctypes.POINTER(DcCfg)], ctypes.c_int64),
    "dc_blob_floats": ([ctypes.POINTER(DcCfg)], ctypes.c_int64),
    "dc_token_buffer": ([_P], _P),
    "dc_audio_buffer": ([_P], _P),
    "dc_f0_buffer": ([_P], _P),
    "dc_get_stats": ([_P, ctypes.POINTER(DcStats)], ctypes.c_int),
    "dc_carry_bytes": ([_P], ctypes.c_int64),
    "dc_carry_export": ([_P, ctypes.c_int32, _P, ctypes.c_size_t], ctypes.c_int),
    "dc_carry_import": ([_P, ctypes.c_int32, _P, ctypes.c_size_t], ctypes.c_int),
    "dc_tap_find": ([_P, ctypes.c_char_p], ctypes.c_int32),
    "dc_tap_read": ([_P, ctypes.c_int32, ctypes.c_int32, ctypes.c_int64, ctypes.c_int32, _P,
                     ctypes.POINTER(ctypes.c_int32)], ctypes.c_int),
    "dc_layer_count": ([_P], ctypes.c_int32),
    "dc_layer_info_get": ([_P, ctypes.c_int32, ctypes.POINTER(DcLayerInfo)], ctypes.c_int),
    "dc_time_layers": ([_P, ctypes.c_int32, ctypes.POINTER(ctypes.c_double)], ctypes.c_int),
    "dc_debug_checks": ([ctypes.c_int32], ctypes.c_int32),
    "dc_last_error": ([_P], ctypes.c_char_p),
    "dc_free": ([_P], None),
}

_lib = None


def lib() -> ctypes.CDLL:
    """The loaded libdc.so; raises if it has not been built."""
    global _lib
    if _lib is None:
        # torch first: libdc.so then binds to the HIP runtime torch has
        # loaded (the same soname), not a second copy of its own
        import torch  # noqa: F401
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with __graft_entry__.build() "
                               "(hipcc --offload-arch=gfx950); there is no fallback path")
        L = ctypes.CDLL(LIB_PATH)
        for name, (args, res) in SIGNATURES.items():
            fn = getattr(L, name)
            fn.argtypes = args
            fn.restype = res
        _lib = L
    return _lib


def make_cfg(arch: dict, dtype: str, batch: int, chunk_tokens: int, max_tokens: int | None = None,
             flags: int = 0, tile_variant: int = 0, stream: int | None = None, rng_seed: int = 0) -> DcCfg:
    c = DcCfg()
    c.abi_version = DC_ABI_VERSION
    c.vocab, c.embed, c.frames_per_token = arch["vocab"], arch["embed"], arch["frames_per_token"]
    c.n_pre, c.pre_kernel = arch["n_pre"], arch["pre_kernel"]
    c.n_stages = len(arch["up_rate"])
    for i, u in enumerate(arch["up_rate"]):
        c.up_rate[i] = u
    for i, ch in enumerate(arch["channels"]):
        c.channels[i] = ch
    c.n_rb = len(arch["rb_kernel"])
    for i, k in enumerate(arch["rb_kernel"]):
        c.rb_kernel[i] = k
    c.n_dil = len(arch["dil"])
    for i, d in enumerate(arch["dil"]):
        c.dil[i] = d
    c.head_kernel, c.n_fft, c.hop = arch["head_kernel"], arch["n_fft"], arch["hop"]
    c.lrelu_slope = arch["lrelu_slope"]
    c.dtype = DC_BF16 if dtype == "bf16" else DC_F32
    c.batch = batch
    c.chunk_tokens = chunk_tokens
    c.max_tokens = max_tokens if max_tokens is not None else chunk_tokens
    c.flags = flags
    c.tile_variant = tile_variant
    c.n_harmonics = arch.get("n_harmonics", 0)
    c.sine_amp = arch.get("sine_amp", 0.0)
    c.noise_std = arch.get("noise_std", 0.0)
    c.voiced_threshold = arch.get("voiced_threshold", 0.0)
    c.sample_rate = arch.get("sample_rate", 0.0)
    c.rng_seed = rng_seed
    c.hip_stream = stream
    return c


def _ptr(x) -> int:
    """Address of a torch tensor (device or host) or a numpy array."""
    if isinstance(x, np.ndarray):
        return x.ctypes.data
    return x.data_ptr()


def _check(status: int, handle) -> int:
    if status != DC_OK:
        raise DcError(status, dc_last_error(handle))
    return status


# ------------------------------------------------------------ the C-ABI calls

def dc_init(blob: np.ndarray, cfg: DcCfg):
    blob = np.ascontiguousarray(blob, dtype=np.float32)
    h = ctypes.c_void_p()
    st = lib().dc_init(blob.ctypes.data, blob.nbytes, ctypes.byref(cfg), ctypes.byref(h))
    if st != DC_OK:
        raise DcError(st, dc_last_error(None))
    return h


def dc_decode_chunk(h, tokens, n: int, audio_out) -> int:
    """Raw call: returns the status (no exception)."""
    return lib().dc_decode_chunk(h, _ptr(tokens) if tokens is not None else None, n,
                                 _ptr(audio_out) if audio_out is not None else None)


def dc_decode_chunk_f0(h, tokens, f0, n: int, audio_out) -> int:
    """Raw call: returns the status (no exception)."""
    return lib().dc_decode_chunk_f0(h, _ptr(tokens) if tokens is not None else None,
                                    _ptr(f0) if f0 is not None else None, n,
                                    _ptr(audio_out) if audio_out is not None else None)


def dc_decode_chunk_f0_static(h, tokens, f0, n: int, audio_out) -> int:
    """Raw call: returns the status (no exception)."""
    return lib().dc_decode_chunk_f0_static(h, _ptr(tokens) if tokens is not None else None,
                                           _ptr(f0) if f0 is not None else None, n,
                                           _ptr(audio_out) if audio_out is not None else None)


def dc_reset(h) -> int:
    return lib().dc_reset(h)


def dc_reset_stream(h, b: int) -> int:
    return lib().dc_reset_stream(h, b)


def dc_sync(h) -> int:
    return lib().dc_sync(h)


def dc_samples_per_token(cfg: DcCfg) -> int:
    return lib().dc_samples_per_token(ctypes.byref(cfg))


def dc_blob_floats(cfg: DcCfg) -> int:
    return lib().dc_blob_floats(ctypes.byref(cfg))


def dc_token_buffer(h) -> int:
    return lib().dc_token_buffer(h)


def dc_audio_buffer(h) -> int:
    return lib().dc_audio_buffer(h)


def dc_f0_buffer(h) -> int:
    return lib().dc_f0_buffer(h)


def dc_carry_bytes(h) -> int:
    return lib().dc_carry_bytes(h)


def dc_carry_export(h, b: int, buf: np.ndarray) -> int:
    """Raw call: fills the uint8 buffer buf (dc_carry_bytes long); returns the status."""
    return lib().dc_carry_export(h, b, buf.ctypes.data, buf.nbytes)


def dc_carry_import(h, b: int, buf: np.ndarray) -> int:
    return lib().dc_carry_import(h, b, buf.ctypes.data, buf.nbytes)


def dc_get_stats(h) -> dict:
    s = DcStats()
    _check(lib().dc_get_stats(h, ctypes.byref(s)), h)
    return s.as_dict()


def dc_tap_find(h, name: str) -> int:
    return lib().dc_tap_find(h, name.encode())


def dc_tap_read(h, tap: int, b: int, frame0: int, nframes: int, channels: int) -> np.ndarray:
    out = np.empty((nframes, channels), dtype=np.float32)
    c = ctypes.c_int32()
    _check(lib().dc_tap_read(h, tap, b, frame0, nframes, out.ctypes.data, ctypes.byref(c)), h)
    assert c.value == channels, (c.value, channels)
    return out


def dc_layer_count(h) -> int:
    return lib().dc_layer_count(h)


def dc_layer_info_get(h, i: int) -> dict:
    info = DcLayerInfo()
    _check(lib().dc_layer_info_get(h, i, ctypes.byref(info)), h)
    return {"name": info.name.decode(), "kernel": info.kernel.decode(), "rows": info.rows,
            "cols": info.cols, "depth": info.depth, "flops": info.flops, "bytes": info.bytes}


def dc_time_layers(h, reps: int) -> list:
    n = dc_layer_count(h)
    buf = (ctypes.c_double * n)()
    _check(lib().dc_time_layers(h, reps, buf), h)
    return list(buf)


def dc_last_error(h) -> str:
    r = lib().dc_last_error(h)
    return r.decode() if r else ""


def dc_free(h) -> None:
    lib().dc_free(h)


# --------------------------------------------------------------- convenience

def _shape_dtype_device(x):
    """(shape, dtype name, device index or None for host memory) of a numpy
    array or a torch tensor."""
    if isinstance(x, np.ndarray):
        return tuple(x.shape), str(x.dtype), None
    dev = x.device
    return tuple(x.shape), str(x.dtype).replace("torch.", ""), (dev.index if dev.type == "cuda" else None)


def check_decode_args(tokens, f0, batch: int, max_tokens: int, fpt: int, has_source: bool, host: bool,
                      device: int | None = 0) -> int:
    """Validate the arguments of Decoder.decode and return n.

    tokens must be [batch][n] with 1 <= n <= max_tokens.  In host mode it is
    a numpy int32 array; in device mode an int32 tensor on the state's device,
    or a numpy array of any integer type whose values fit int32 (copied).  A
    decoder with a harmonic source needs f0 [batch][n * fpt] float32 in the
    same form (numpy float arrays are converted).  Anything else raises
    DcError: DC_ERANGE for n > max_tokens (the status the C call gives), else
    DC_EINVAL.  The C call reads tokens as int32 and trusts the row count, so
    an int64 tensor or a short one would otherwise be misread silently."""
    if tokens is None:
        raise DcError(DC_EINVAL, "tokens is None")
    shape, dt, dev = _shape_dtype_device(tokens)
    if len(shape) != 2 or shape[0] != batch:
        raise DcError(DC_EINVAL, f"tokens must be [batch={batch}][n], got shape {shape}")
    n = shape[1]
    if n < 1:
        raise DcError(DC_EINVAL, f"n = {n} tokens per stream; at least 1 is needed")
    if n > max_tokens:
        raise DcError(DC_ERANGE, f"n = {n} tokens per stream exceeds max_tokens = {max_tokens}")
    if isinstance(tokens, np.ndarray):
        if host and dt != "int32":
            raise DcError(DC_EINVAL, f"host-mode tokens must be int32, got {dt}")
        if not np.issubdtype(tokens.dtype, np.integer):
            raise DcError(DC_EINVAL, f"tokens must be integers, got {dt}")
        if tokens.size and (int(tokens.min()) < -2 ** 31 or int(tokens.max()) >= 2 ** 31):
            raise DcError(DC_EINVAL, "token ids do not fit int32")
    else:
        if host:
            raise DcError(DC_EINVAL, "host-mode tokens must be a numpy int32 array")
        if dt != "int32":
            raise DcError(DC_EINVAL, f"device tokens must be an int32 tensor, got {dt}")
        if dev is None or (device is not None and dev != device):
            raise DcError(DC_EINVAL, f"device tokens must live on cuda:{device}, got {tokens.device}")
    if has_source:
        if f0 is None:
            raise DcError(DC_EINVAL, "a decoder with a harmonic source needs f0")
        fshape, fdt, fdev = _shape_dtype_device(f0)
        if fshape != (batch, n * fpt):
            raise DcError(DC_EINVAL, f"f0 must be [batch={batch}][n*frames_per_token={n * fpt}], got {fshape}")
        if isinstance(f0, np.ndarray):
            if host and fdt != "float32":
                raise DcError(DC_EINVAL, f"host-mode f0 must be float32, got {fdt}")
            if not np.issubdtype(f0.dtype, np.floating):
                raise DcError(DC_EINVAL, f"f0 must be floating point, got {fdt}")
        else:
            if host:
                raise DcError(DC_EINVAL, "host-mode f0 must be a numpy float32 array")
            if fdt != "float32":
                raise DcError(DC_EINVAL, f"device f0 must be a float32 tensor, got {fdt}")
            if fdev is None or (device is not None and fdev != device):
                raise DcError(DC_EINVAL, f"device f0 must live on cuda:{device}, got {f0.device}")
    elif f0 is not None:
        raise DcError(DC_EINVAL, "f0 given to a decoder without a harmonic source")
    return n


class Decoder:
    """One dc_state on the current GPU, with torch-ROCm tensors for device memory
    and a dedicated torch stream that every call is ordered on."""

    def __init__(self, arch: dict, dtype: str, blob: np.ndarray, batch: int, chunk_tokens: int,
                 max_tokens: int | None = None, flags: int = 0, tile_variant: int = 0, rng_seed: int = 0):
        import torch
        self.torch = torch
        self.arch, self.dtype, self.batch = arch, dtype, batch
        self.host = bool(flags & DC_HOST_PTRS)
        self.stream = torch.cuda.Stream()
        self.cfg = make_cfg(arch, dtype, batch, chunk_tokens, max_tokens, flags, tile_variant,
                            self.stream.cuda_stream, rng_seed)
        self.has_source = arch.get("n_harmonics", 0) > 0
        self.spt = dc_samples_per_token(self.cfg)
        self.chunk_tokens = chunk_tokens
        self.max_tokens = self.cfg.max_tokens
        self.h = dc_init(blob, self.cfg)

    def close(self):
        if self.h is not None:
            dc_free(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def decode(self, tokens, f0=None, check: bool = True, static_scratch: bool = False):
        """tokens [batch][n] int32 (numpy in host mode, else a device tensor or
        numpy copied to the device), and for a decoder with a harmonic source
        f0 [batch][n*frames_per_token] float32 likewise -> PCM [batch][n*spt]
        (numpy in host mode, else a device tensor).  Arguments that the C call
        would misread (another dtype, rank, row count or device) raise DcError
        before anything is launched; see check_decode_args.  static_scratch
        (a decoder with a harmonic source) calls dc_decode_chunk_f0_static."""
        torch = self.torch
        n = check_decode_args(tokens, f0, self.batch, self.max_tokens, self.arch["frames_per_token"],
                              self.has_source, self.host, torch.cuda.current_device())
        if self.host:
            tok = np.ascontiguousarray(tokens, dtype=np.int32)
            out = np.empty((self.batch, n * self.spt), dtype=np.float32)
            if self.has_source:
                call = dc_decode_chunk_f0_static if static_scratch else dc_decode_chunk_f0
                st = call(self.h, tok, np.ascontiguousarray(f0, dtype=np.float32), n, out)
            else:
                st = dc_decode_chunk(self.h, tok, n, out)
        else:
            with torch.cuda.stream(self.stream):
                if isinstance(tokens, np.ndarray):
                    tok = torch.from_numpy(np.ascontiguousarray(tokens, dtype=np.int32)).to("cuda")
                else:
                    tok = tokens.contiguous()
                f0d = None
                if self.has_source and f0 is not None:
                    if isinstance(f0, np.ndarray):
                        f0d = torch.from_numpy(np.ascontiguousarray(f0, dtype=np.float32)).to("cuda")
                    else:
                        f0d = f0.contiguous()
                out = torch.empty((self.batch, n * self.spt), dtype=torch.float32, device="cuda")
            self.stream.wait_stream(torch.cuda.current_stream())
            if self.has_source:
                call = dc_decode_chunk_f0_static if static_scratch else dc_decode_chunk_f0
                st = call(self.h, tok, f0d, n, out)
            else:
                st = dc_decode_chunk(self.h, tok, n, out)
            tok.record_stream(self.stream)
            if f0d is not None:
                f0d.record_stream(self.stream)
            out.record_stream(self.stream)
            torch.cuda.current_stream().wait_stream(self.stream)
        if check:
            _check(st, self.h)
        return out

    def sync(self):
        return _check(dc_sync(self.h), self.h)

    def reset(self):
        return _check(dc_reset(self.h), self.h)

    def reset_stream(self, b: int):
        return _check(dc_reset_stream(self.h, b), self.h)

    def stats(self) -> dict:
        return dc_get_stats(self.h)

    def export_carry(self, b: int) -> np.ndarray:
        """Snapshot of stream b's carry (host bytes)."""
        buf = np.empty(dc_carry_bytes(self.h), dtype=np.uint8)
        _check(dc_carry_export(self.h, b, buf), self.h)
        return buf

    def import_carry(self, b: int, snap: np.ndarray):
        """Continue the snapshot's stream in stream b of this state."""
        return _check(dc_carry_import(self.h, b, np.ascontiguousarray(snap, dtype=np.uint8)), self.h)

    def layers(self) -> list:
        return [dc_layer_info_get(self.h, i) for i in range(dc_layer_count(self.h))]

    def time_layers(self, reps: int) -> list:
        return dc_time_layers(self.h, reps)

    def tap(self, name: str, b: int, frame0: int, nframes: int) -> np.ndarray:
        t = dc_tap_find(self.h, name)
        if t < 0:
            raise KeyError(name)
        ch = _tap_channels(self.arch, name)
        return dc_tap_read(self.h, t, b, frame0, nframes, ch)


def _tap_channels(arch: dict, name: str) -> int:
    if name == "embed" or name.startswith("pre"):
        return arch["channels"][0]
    if name == "head":
        return 2 * (arch["n_fft"] // 2 + 1)
    if name == "G":
        return arch["n_fft"]
    if name == "src":
        return arch["hop"]
    s = int(name[1:name.index(".")])
    return arch["channels"][s + 1]
