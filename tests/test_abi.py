"""The C-ABI library on the host: it loads, exports every symbol that
include/dc.h and include/dc_flow.h declare, and its host-only logic (sizes,
configuration checks) fails closed before touching the device.  No GPU
needed."""
import ctypes
import os
import re

import numpy as np
import pytest

import paper_2609_35115_amd as dc
from paper_2609_35115_amd import flow, synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_functions(header: str | None = None):
    names = set()
    for h in ([header] if header else sorted(os.listdir(os.path.join(ROOT, "include")))):
        if not h.endswith(".h"):
            continue
        text = open(os.path.join(ROOT, "include", h)).read()
        text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
        names |= set(re.findall(r"\b(dc_[a-z0-9_]+)\s*\(", text))
    return sorted(names)


def test_header_and_binding_agree():
    assert declared_functions("dc.h") == sorted(dc.SIGNATURES)
    assert declared_functions("dc_flow.h") == sorted(flow.FLOW_SIGNATURES)
    assert declared_functions() == sorted(set(dc.SIGNATURES) | set(flow.FLOW_SIGNATURES))


def test_library_exports_every_declared_symbol():
    L = ctypes.CDLL(dc.LIB_PATH)
    for name in declared_functions():
        assert hasattr(L, name), name


def test_struct_sizes_match_header_layout():
    # dc_cfg: 34 int32 fields + float + uint32 (144 bytes), the source's int32
    # and four floats (164, padded to 168), the uint64 seed and the pointer
    assert ctypes.sizeof(dc.DcCfg) == 168 + 8 + 8
    # dc_stats: 12 int64, 2 int32, a double, then replays_flush, two int32, staged_f0 and direct_static
    assert ctypes.sizeof(dc.DcStats) == 12 * 8 + 2 * 4 + 8 + 8 + 2 * 4 + 8 + 8


@pytest.mark.parametrize("name", list(synth.WORKLOADS))
def test_sizes_agree_with_generator(name):
    w = synth.workload(name)
    cfg = dc.make_cfg(w["arch"], w["dtype"], w["batch"], w["chunk_tokens"])
    assert dc.dc_samples_per_token(cfg) == synth.samples_per_token(w["arch"])
    assert dc.dc_blob_floats(cfg) == synth.blob_floats(w["arch"])


def _init_status(cfg, blob):
    blob = np.ascontiguousarray(blob, dtype=np.float32)
    h = ctypes.c_void_p()
    st = dc.lib().dc_init(blob.ctypes.data, blob.nbytes, ctypes.byref(cfg), ctypes.byref(h))
    return st, h.value


def test_init_rejects_bad_configs_before_any_device_call():
    arch = synth.TINY_ARCH
    blob = synth.make_weights(arch)
    good = lambda **kw: dc.make_cfg(arch, "f32", kw.pop("batch", 1), kw.pop("chunk", 8), kw.pop("max", 8))
    c = good()
    c.abi_version = 99
    assert _init_status(c, blob) == (dc.DC_EVERSION, None)
    c = good()
    c.n_fft = 32
    assert _init_status(c, blob)[0] == dc.DC_EINVAL
    assert "n_fft" in dc.dc_last_error(None)
    c = good(chunk=9, max=8)
    assert _init_status(c, blob)[0] == dc.DC_EINVAL
    c = good()
    c.channels[2] = 12
    assert _init_status(c, blob)[0] == dc.DC_EINVAL
    c = good()
    c.dtype = 7
    assert _init_status(c, blob)[0] == dc.DC_EINVAL
    c = good()
    c.flags = 1 << 7
    assert _init_status(c, blob)[0] == dc.DC_EINVAL
    c = good()
    c.flags = dc.DC_FLUSH_CATALOG | dc.DC_NO_GRAPH   # a catalog needs graphs
    assert _init_status(c, blob)[0] == dc.DC_EINVAL
    assert "DC_FLUSH_CATALOG" in dc.dc_last_error(None)
    c = good()
    assert _init_status(c, blob[:-1])[0] == dc.DC_EINVAL
    assert "blob size" in dc.dc_last_error(None)
    # the harmonic source: its blob holds the extra tensors, its fields are checked
    nsf = synth.TINY_NSF_ARCH
    nblob = synth.make_weights(nsf)
    c = dc.make_cfg(nsf, "f32", 1, 8, 8)
    assert dc.dc_blob_floats(c) == synth.blob_floats(nsf) == blob.size + (nsf["n_harmonics"] + 2) + 8 * 5
    assert _init_status(c, blob)[0] == dc.DC_EINVAL            # the source tensors are missing
    c.n_harmonics = 40
    assert _init_status(c, nblob)[0] == dc.DC_EINVAL
    c = dc.make_cfg(nsf, "f32", 1, 8, 8)
    c.sample_rate = 0.0
    assert _init_status(c, nblob)[0] == dc.DC_EINVAL
    assert "sample_rate" in dc.dc_last_error(None)


def test_null_state_calls_fail_closed():
    L = dc.lib()
    assert L.dc_decode_chunk(None, None, 1, None) == dc.DC_EINVAL
    assert L.dc_decode_chunk_f0(None, None, None, 1, None) == dc.DC_EINVAL
    assert L.dc_decode_chunk_f0_static(None, None, None, 1, None) == dc.DC_EINVAL
    assert L.dc_f0_buffer(None) is None
    assert L.dc_carry_bytes(None) == 0
    assert L.dc_carry_export(None, 0, None, 0) == dc.DC_EINVAL
    assert L.dc_carry_import(None, 0, None, 0) == dc.DC_EINVAL
    assert L.dc_reset(None) == dc.DC_EINVAL
    assert L.dc_sync(None) == dc.DC_EINVAL
    assert L.dc_token_buffer(None) is None
    assert L.dc_tap_find(None, b"embed") == -1
    L.dc_free(None)


# ------------------------------------------------------------ flow decoder

def test_flow_struct_sizes_match_header_layout():
    # 14 int32 + uint32 flags + two floats (68, padded to 72), the seed, the stream
    assert ctypes.sizeof(flow.DcFlowCfg) == 72 + 8 + 8
    # 9 int64, 2 int32, a double
    assert ctypes.sizeof(flow.DcFlowStats) == 9 * 8 + 2 * 4 + 8
    # a 48-byte name, 2 int32, 3 doubles
    assert ctypes.sizeof(flow.DcFlowKernelStat) == 48 + 8 + 24


@pytest.mark.parametrize("arch", [synth.TINY_FLOW_ARCH, synth.REAL_FLOW_ARCH])
def test_flow_blob_size_agrees_with_generator(arch):
    assert flow.dc_flow_blob_floats(flow.make_flow_cfg(arch, "bf16", 4)) == synth.flow_blob_floats(arch)


def _flow_init_status(cfg, blob):
    blob = np.ascontiguousarray(blob, dtype=np.float32)
    h = ctypes.c_void_p()
    st = flow.flib().dc_flow_init(blob.ctypes.data, blob.nbytes, ctypes.byref(cfg), ctypes.byref(h))
    return st, h.value


def test_flow_init_rejects_bad_configs_before_any_device_call():
    arch = synth.TINY_FLOW_ARCH
    blob = synth.make_flow_weights(arch)
    good = lambda: flow.make_flow_cfg(arch, "f32", 2)
    c = good()
    c.abi_version = 7
    assert _flow_init_status(c, blob) == (dc.DC_EVERSION, None)
    for field, value, words in [("heads", 3, "dim"), ("n_mel", 12, "n_mel"), ("mlp", 100, "mlp"),
                                ("f_call", 7, "f_chunk"), ("f_retained", 12, "f_retained"),
                                ("dtype", 5, "dtype"), ("flags", 64, "flags"), ("batch", 0, "batch"),
                                ("t_dim", 3, "t_dim")]:
        c = good()
        setattr(c, field, value)
        assert _flow_init_status(c, blob)[0] == dc.DC_EINVAL, field
        assert words in flow.dc_flow_last_error(None), (field, flow.dc_flow_last_error(None))
        assert flow.dc_flow_blob_floats(c) == 0
    assert _flow_init_status(good(), blob[:-1])[0] == dc.DC_EINVAL
    assert "blob size" in flow.dc_flow_last_error(None)


def test_flow_null_state_calls_fail_closed():
    L = flow.flib()
    assert L.dc_flow_prompt(None, 0, None, None, None, 1) == dc.DC_EINVAL
    assert L.dc_flow_decode_chunk(None, None, 1, None) == dc.DC_EINVAL
    assert L.dc_flow_sync(None) == dc.DC_EINVAL
    assert L.dc_flow_carry_read(None, 0, 0, 0, 0, 0, None, None) == dc.DC_EINVAL
    assert L.dc_flow_get_stats(None, None) == dc.DC_EINVAL
    assert L.dc_flow_blob_floats(None) == 0
    assert L.dc_flow_profile(None, 1, None, 0, None) == dc.DC_EINVAL
    L.dc_flow_free(None)
