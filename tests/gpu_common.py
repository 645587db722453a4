"""Shared helpers of the GPU tests (no test functions here)."""
from __future__ import annotations

import os
import sys

import numpy as np

import oracle
from paper_2609_35115_amd import synth

TOL = {"f32": 1e-4, "bf16": 2e-2}

# Lead-in tokens before a sampled window: more than the decoder's receptive
# field (about 19 tokens for the real architecture, 4 for the tiny one), so the
# oracle decoding [start - LEAD, end) from the zero state reproduces the
# samples of [start, end) exactly (pinned by test_finite_receptive_field_window).
LEAD = 25


def say(msg: str) -> None:
    print(msg, flush=True)
    sys.stdout.flush()


def err_stats(y: np.ndarray, ref: np.ndarray) -> tuple[float, float]:
    """(max-abs-error / RMS(ref), RMS(error) / RMS(ref))."""
    y = np.asarray(y, dtype=np.float64)
    rms = float(np.sqrt(np.mean(ref ** 2)))
    d = y - ref
    return float(np.abs(d).max() / rms), float(np.sqrt(np.mean(d ** 2)) / rms)


def oracle_window(arch, dtype, blob, ids_stream, start_tok, end_tok):
    """Oracle PCM of tokens [start_tok, end_tok) of one stream (decoded from
    max(0, start_tok - LEAD))."""
    spt = synth.samples_per_token(arch)
    s0 = max(0, start_tok - LEAD)
    pcm = oracle.decode(arch, dtype, blob, ids_stream[s0:end_tok])
    return pcm[(start_tok - s0) * spt:]


def bits_equal(a: np.ndarray, b: np.ndarray) -> bool:
    a = np.ascontiguousarray(a, dtype=np.float32)
    b = np.ascontiguousarray(b, dtype=np.float32)
    return a.shape == b.shape and np.array_equal(a.view(np.uint32), b.view(np.uint32))
