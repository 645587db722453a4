"""Python binding of the flow-decoder calls of libdc.so (include/dc_flow.h).

Argument marshalling only: every step of the chunk call runs in the gfx950
kernels of libdc.so.  There is no fallback: if the library is missing,
loading raises.
"""
from __future__ import annotations

import ctypes

import numpy as np

from . import DC_BF16, DC_F32, DC_HOST_PTRS, DC_NO_GRAPH, DC_OK, DcError, _ptr, lib  # noqa: F401

DC_FLOW_ABI_VERSION = 1
_P = ctypes.c_void_p


class DcFlowCfg(ctypes.Structure):
    _fields_ = [
        ("abi_version", ctypes.c_int32),
        ("n_mel", ctypes.c_int32), ("dim", ctypes.c_int32), ("heads", ctypes.c_int32), ("depth", ctypes.c_int32),
        ("mlp", ctypes.c_int32), ("t_dim", ctypes.c_int32), ("n_steps", ctypes.c_int32),
        ("f_prompt", ctypes.c_int32), ("f_retained", ctypes.c_int32), ("f_chunk", ctypes.c_int32),
        ("f_call", ctypes.c_int32), ("batch", ctypes.c_int32), ("dtype", ctypes.c_int32),
        ("flags", ctypes.c_uint32), ("cfg_rate", ctypes.c_float), ("temperature", ctypes.c_float),
        ("rng_seed", ctypes.c_uint64), ("hip_stream", ctypes.c_void_p),
    ]


class DcFlowStats(ctypes.Structure):
    _fields_ = [
        ("calls", ctypes.c_int64), ("replays", ctypes.c_int64), ("direct", ctypes.c_int64),
        ("prompts", ctypes.c_int64), ("rejected", ctypes.c_int64), ("weight_bytes", ctypes.c_int64),
        ("carry_bytes", ctypes.c_int64), ("carry_live_bytes", ctypes.c_int64), ("arena_bytes", ctypes.c_int64),
        ("kernels_per_call", ctypes.c_int32), ("graph_nodes", ctypes.c_int32), ("capture_ms", ctypes.c_double),
    ]


class DcFlowKernelStat(ctypes.Structure):
    _fields_ = [
        ("name", ctypes.c_char * 48), ("launches", ctypes.c_int32), ("mfma", ctypes.c_int32),
        ("us", ctypes.c_double), ("flops", ctypes.c_double), ("bytes", ctypes.c_double),
    ]


FLOW_SIGNATURES = {
    "dc_flow_blob_floats": ([ctypes.POINTER(DcFlowCfg)], ctypes.c_int64),
    "dc_flow_init": ([_P, ctypes.c_size_t, ctypes.POINTER(DcFlowCfg), ctypes.POINTER(_P)], ctypes.c_int),
    "dc_flow_prompt": ([_P, ctypes.c_int32, _P, _P, _P, ctypes.c_int32], ctypes.c_int),
    "dc_flow_decode_chunk": ([_P, _P, ctypes.c_int32, _P], ctypes.c_int),
    "dc_flow_sync": ([_P], ctypes.c_int),
    "dc_flow_carry_read": ([_P, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, _P,
                            ctypes.POINTER(ctypes.c_int32)], ctypes.c_int),
    "dc_flow_get_stats": ([_P, ctypes.POINTER(DcFlowStats)], ctypes.c_int),
    "dc_flow_profile": ([_P, ctypes.c_int32, ctypes.POINTER(DcFlowKernelStat), ctypes.c_int32,
                         ctypes.POINTER(ctypes.c_int32)], ctypes.c_int),
    "dc_flow_last_error": ([_P], ctypes.c_char_p),
    "dc_flow_free": ([_P], None),
}

_bound = False


def flib() -> ctypes.CDLL:
    global _bound
    L = lib()
    if not _bound:
        for name, (args, res) in FLOW_SIGNATURES.items():
            fn = getattr(L, name)
            fn.argtypes = args
            fn.restype = res
        _bound = True
    return L


def make_flow_cfg(arch: dict, dtype: str, batch: int, flags: int = 0, stream: int | None = None,
                  rng_seed: int = 0) -> DcFlowCfg:
    c = DcFlowCfg()
    c.abi_version = DC_FLOW_ABI_VERSION
    for name in ("n_mel", "dim", "heads", "depth", "mlp", "t_dim", "n_steps", "f_prompt", "f_retained", "f_chunk",
                 "f_call"):
        setattr(c, name, arch[name])
    c.cfg_rate, c.temperature = arch["cfg_rate"], arch["temperature"]
    c.batch = batch
    c.dtype = DC_BF16 if dtype == "bf16" else DC_F32
    c.flags = flags
    c.rng_seed = rng_seed
    c.hip_stream = stream
    return c


def dc_flow_last_error(h) -> str:
    msg = flib().dc_flow_last_error(h)
    return msg.decode() if msg else ""


def _check(status: int, h) -> int:
    if status != DC_OK:
        raise DcError(status, dc_flow_last_error(h))
    return status


def dc_flow_blob_floats(cfg: DcFlowCfg) -> int:
    return int(flib().dc_flow_blob_floats(ctypes.byref(cfg)))


def dc_flow_init(blob: np.ndarray, cfg: DcFlowCfg):
    blob = np.ascontiguousarray(blob, dtype=np.float32)
    h = ctypes.c_void_p()
    st = flib().dc_flow_init(blob.ctypes.data, blob.nbytes, ctypes.byref(cfg), ctypes.byref(h))
    if st != DC_OK:
        raise DcError(st, dc_flow_last_error(None))
    return h


def dc_flow_prompt(h, b: int, mu, cond, spk, frames: int) -> int:
    """Raw call: returns the status (no exception)."""
    return flib().dc_flow_prompt(h, b, _ptr(mu) if mu is not None else None, _ptr(cond) if cond is not None else None,
                                 _ptr(spk) if spk is not None else None, frames)


def dc_flow_decode_chunk(h, mu, n: int, mel_out) -> int:
    """Raw call: returns the status (no exception)."""
    return flib().dc_flow_decode_chunk(h, _ptr(mu) if mu is not None else None, n,
                                       _ptr(mel_out) if mel_out is not None else None)


def dc_flow_sync(h) -> int:
    return flib().dc_flow_sync(h)


def dc_flow_carry_read(h, b: int, step: int, layer: int, branch: int, kv: int, dim: int) -> np.ndarray:
    frames = ctypes.c_int32()
    _check(flib().dc_flow_carry_read(h, b, step, layer, branch, kv, None, ctypes.byref(frames)), h)
    out = np.empty((frames.value, dim), dtype=np.float32)
    if frames.value:
        _check(flib().dc_flow_carry_read(h, b, step, layer, branch, kv, out.ctypes.data, ctypes.byref(frames)), h)
    return out


def dc_flow_get_stats(h) -> dict:
    s = DcFlowStats()
    _check(flib().dc_flow_get_stats(h, ctypes.byref(s)), h)
    return {name: getattr(s, name) for name, _ in DcFlowStats._fields_}


def dc_flow_profile(h, reps: int) -> list:
    """Per-role device time of one f_call-frame call (dicts, in launch order of first use)."""
    n = ctypes.c_int32()
    _check(flib().dc_flow_profile(h, reps, None, 0, ctypes.byref(n)), h)
    arr = (DcFlowKernelStat * n.value)()
    _check(flib().dc_flow_profile(h, reps, arr, n.value, ctypes.byref(n)), h)
    return [{"name": a.name.decode(), "launches": a.launches, "mfma": bool(a.mfma), "us": a.us,
             "flops": a.flops, "bytes": a.bytes} for a in arr]


def dc_flow_free(h) -> None:
    flib().dc_flow_free(h)


class FlowDecoder:
    """One dc_flow_state on the current GPU; device memory from torch-ROCm,
    every call ordered on a dedicated torch stream."""

    def __init__(self, arch: dict, dtype: str, blob: np.ndarray, batch: int, flags: int = 0, rng_seed: int = 0):
        import torch
        self.torch = torch
        self.arch, self.dtype, self.batch = dict(arch), dtype, batch
        self.host = bool(flags & DC_HOST_PTRS)
        self.stream = torch.cuda.Stream()
        self.cfg = make_flow_cfg(arch, dtype, batch, flags, self.stream.cuda_stream, rng_seed)
        self.h = dc_flow_init(blob, self.cfg)

    def close(self):
        if self.h is not None:
            dc_flow_free(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def _dev(self, a):
        torch = self.torch
        if isinstance(a, np.ndarray):
            return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to("cuda")
        return a.contiguous()

    def prompt(self, b: int, mu, cond, spk):
        """Start a turn of stream b: mu, cond [frames][n_mel], spk [n_mel]."""
        torch = self.torch
        frames = mu.shape[0]
        if self.host:
            args = [np.ascontiguousarray(x, dtype=np.float32) for x in (mu, cond, spk)]
            return _check(dc_flow_prompt(self.h, b, *args, frames), self.h)
        with torch.cuda.stream(self.stream):
            args = [self._dev(x) for x in (mu, cond, spk)]
        self.stream.wait_stream(torch.cuda.current_stream())
        st = dc_flow_prompt(self.h, b, *args, frames)
        for x in args:
            x.record_stream(self.stream)
        torch.cuda.current_stream().wait_stream(self.stream)
        return _check(st, self.h)

    def decode(self, mu, check: bool = True):
        """mu [batch][n][n_mel] -> mel [batch][n][n_mel] (numpy in host mode,
        else a device tensor)."""
        torch = self.torch
        n = mu.shape[1]
        M = self.arch["n_mel"]
        if self.host:
            out = np.empty((self.batch, n, M), dtype=np.float32)
            st = dc_flow_decode_chunk(self.h, np.ascontiguousarray(mu, dtype=np.float32), n, out)
        else:
            with torch.cuda.stream(self.stream):
                mud = self._dev(mu)
                out = torch.empty((self.batch, n, M), dtype=torch.float32, device="cuda")
            self.stream.wait_stream(torch.cuda.current_stream())
            st = dc_flow_decode_chunk(self.h, mud, n, out)
            mud.record_stream(self.stream)
            out.record_stream(self.stream)
            torch.cuda.current_stream().wait_stream(self.stream)
        if check:
            _check(st, self.h)
        return out

    def sync(self):
        return _check(dc_flow_sync(self.h), self.h)

    def carry(self, b: int, step: int, layer: int, branch: int, kv: int) -> np.ndarray:
        return dc_flow_carry_read(self.h, b, step, layer, branch, kv, self.arch["dim"])

    def stats(self) -> dict:
        return dc_flow_get_stats(self.h)

    def profile(self, reps: int = 5) -> list:
        return dc_flow_profile(self.h, reps)
