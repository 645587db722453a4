"""Seeded synthetic workloads: decoder architectures, random weights and token ids.

This module holds no arithmetic of the decode step.  It only describes the
shapes of the streaming Token2Wav vocoder workloads and draws the random
numbers they are fed with, so that the GPU library and the CPU oracle can be
driven with identical inputs.

Workload shapes follow the paper's shared streaming decoder (Evaluation,
"Setup"): 25 Hz speech tokens, 2 frames per token, 25-token chunks that each
become one second of 24 kHz PCM, and several independent sessions sharing one
set of weights (Design, "Why the two rules are inseparable", multi-session
paragraph).  The paper publishes no layer shapes and no weights, so the
architectures below are synthetic random-weight decoders of that shape.

Weight blob format (little-endian float32, tensors back to back, PyTorch
layouts):

    emb              [vocab][embed]
    per pre layer:   W [C0][C0][pre_kernel], b [C0]
    per stage s:     convT W [C_{s-1}][C_s][2*u_s], b [C_s]
                     per resblock kernel k_j, per dilation d:
                         W1 [C_s][C_s][k_j], b1 [C_s], W2 [C_s][C_s][k_j], b2 [C_s]
    head:            W [2*(n_fft/2+1)][C_last][head_kernel], b [2*(n_fft/2+1)]
    harmonic source (architectures with n_harmonics > 0 only):
                     merge W [n_harmonics+1], merge b [1],
                     down W [C_last][1][hop], down b [C_last]

Weights are N(0, 1/fan_in) with fan_in = C_in*k for a Conv1d and 2*C_in for a
ConvTranspose1d with kernel 2u and stride u (each output reads two input
frames); biases are N(0, 1/fan_in) of their layer; the embedding is N(0, 1).
All draws come from numpy's PCG64 seeded by SeedSequence([seed, 0]) in blob
order, in float64, then rounded to float32.  Token ids of stream b come from
SeedSequence([seed, 1, b]), uniform over the vocabulary.

The harmonic source takes a fundamental frequency per frame of the pre-stack
clock (f0, Hz; 0 where unvoiced).  Its synthetic contour for stream b comes
from SeedSequence([seed, 2, b]): alternating unvoiced and voiced runs of
geometric length (means 8 and 24 frames, i.e. 0.16 s and 0.48 s at 50 Hz),
voiced frames following a per-stream base pitch in [90, 250] Hz times
2^(w/12) for a random walk w of N(0, 0.25) semitone steps, clipped to
[60, 500] Hz -- the range of speech.
"""
from __future__ import annotations

import copy
import math

import numpy as np

TINY_ARCH = dict(
    vocab=256, embed=64, frames_per_token=1,
    n_pre=4, pre_kernel=3,
    up_rate=[2, 2, 4], channels=[64, 32, 16, 8],
    rb_kernel=[3], dil=[1, 3],
    head_kernel=7, n_fft=16, hop=4, lrelu_slope=0.1,
)

REAL_ARCH = dict(
    vocab=6561, embed=512, frames_per_token=2,
    n_pre=8, pre_kernel=3,
    up_rate=[8, 5, 3], channels=[512, 256, 128, 64],
    rb_kernel=[3, 7, 11], dil=[1, 3, 5],
    head_kernel=7, n_fft=16, hop=4, lrelu_slope=0.1,
)

# The same decoders with the harmonic-plus-noise excitation source: the
# fundamental and n_harmonics overtones, sine amplitude 0.1, noise 0.003 on
# voiced frames (amplitude / 3 on unvoiced ones), voiced above 10 Hz.
_SOURCE = dict(sine_amp=0.1, noise_std=0.003, voiced_threshold=10.0, sample_rate=24000.0)
TINY_NSF_ARCH = dict(TINY_ARCH, n_harmonics=2, **_SOURCE)
REAL_NSF_ARCH = dict(REAL_ARCH, n_harmonics=8, **_SOURCE)

# Workloads: architecture, arithmetic type, independent streams, tokens per
# chunk and chunks per measured pass.
WORKLOADS = {
    "tiny_f32_b1_n8": dict(arch=TINY_ARCH, dtype="f32", batch=1, chunk_tokens=8, chunks=8),
    "real_f32_b1_n25": dict(arch=REAL_ARCH, dtype="f32", batch=1, chunk_tokens=25, chunks=20),
    "real_bf16_b16_n25": dict(arch=REAL_ARCH, dtype="bf16", batch=16, chunk_tokens=25, chunks=20),
    "real_bf16_b1_n4": dict(arch=REAL_ARCH, dtype="bf16", batch=1, chunk_tokens=4, chunks=200),
    "real_bf16_b128_n25": dict(arch=REAL_ARCH, dtype="bf16", batch=128, chunk_tokens=25, chunks=40),
}

# The harmonic source's workloads (f0 given per frame, see make_f0).
NSF_WORKLOADS = {
    "real_f32_b1_n25_nsf": dict(arch=REAL_NSF_ARCH, dtype="f32", batch=1, chunk_tokens=25, chunks=20),
    "real_bf16_b16_n25_nsf": dict(arch=REAL_NSF_ARCH, dtype="bf16", batch=16, chunk_tokens=25, chunks=20),
}

SAMPLE_RATE = 24000  # output rate of the real architecture (960 samples / 25 Hz token)

# ---------------------------------------------------------------------------
# Flow decoder (conditional flow matching with a DiT velocity estimator), the
# stage before the vocoder in the Token2Wav pipeline.  The clock quantities
# are the paper's adapter declaration (Design, "Adapter"; Table S11):
# f_prompt = 302, f_retained = 100, f_chunk = 50 and f_call = 56 frames,
# n_steps = 10 solver steps, each evaluating the estimator on the
# conditional and the unconditional input (classifier-free guidance x2).
# The paper gives no layer shapes; it gives the stacked carry's declared
# live size, 0.125 MiB per frame in fp32 (Table 2), which a 16-block DiT of
# width 512 with both guidance branches holds exactly: 16 blocks x (K, V) x
# 512 x 2 branches x 4 bytes.  The rest (8 heads of 64, MLP 2048, 80 mel
# bins, a 256-wide sinusoidal time embedding) is the common DiT shape.
#
# Weight blob (float32, PyTorch Linear layouts [out][in], back to back):
#
#     t.W1 [dim][t_dim], t.b1 [dim], t.W2 [dim][dim], t.b2 [dim]
#     in.W [dim][4*n_mel], in.b [dim]          (input = x | mu | spk | cond)
#     per block l: ada.W [6*dim][dim], ada.b [6*dim],
#                  qkv.W [3*dim][dim], qkv.b [3*dim], o.W [dim][dim], o.b [dim],
#                  fc1.W [mlp][dim], fc1.b [mlp], fc2.W [dim][mlp], fc2.b [dim]
#     final:       ada.W [2*dim][dim], ada.b [2*dim], out.W [n_mel][dim], out.b [n_mel]
#
# drawn like the vocoder's blob (N(0, 1/fan_in), fan_in = in-features, from
# SeedSequence([seed, 0]) in blob order).
TINY_FLOW_ARCH = dict(
    n_mel=16, dim=128, heads=2, depth=2, mlp=256, t_dim=32, n_steps=4,
    f_prompt=20, f_retained=16, f_chunk=8, f_call=11, cfg_rate=0.7, temperature=1.0,
)
REAL_FLOW_ARCH = dict(
    n_mel=80, dim=512, heads=8, depth=16, mlp=2048, t_dim=256, n_steps=10,
    f_prompt=302, f_retained=100, f_chunk=50, f_call=56, cfg_rate=0.7, temperature=1.0,
)

# Flow workloads: architecture, arithmetic type, streams, chunks per pass.
# Every call presents f_call frames (f_chunk retained plus the lookahead).
FLOW_WORKLOADS = {
    "flow_tiny_f32_b2": dict(arch=TINY_FLOW_ARCH, dtype="f32", batch=2, chunks=6),
    "flow_real_f32_b1": dict(arch=REAL_FLOW_ARCH, dtype="f32", batch=1, chunks=6),
    "flow_real_bf16_b1": dict(arch=REAL_FLOW_ARCH, dtype="bf16", batch=1, chunks=6),
    "flow_real_bf16_b16": dict(arch=REAL_FLOW_ARCH, dtype="bf16", batch=16, chunks=6),
    "flow_real_bf16_b128": dict(arch=REAL_FLOW_ARCH, dtype="bf16", batch=128, chunks=6),
}


def workload(name: str) -> dict:
    """Deep copy of a named workload description."""
    for table in (WORKLOADS, NSF_WORKLOADS, FLOW_WORKLOADS):
        if name in table:
            return copy.deepcopy(table[name])
    raise KeyError(name)


def head_channels(arch: dict) -> int:
    return 2 * (arch["n_fft"] // 2 + 1)


def samples_per_token(arch: dict) -> int:
    return arch["frames_per_token"] * math.prod(arch["up_rate"]) * arch["hop"]


def tensor_list(arch: dict):
    """(name, shape, fan_in) for every tensor of the blob, in blob order."""
    out = []
    c0 = arch["channels"][0]
    out.append(("emb", (arch["vocab"], arch["embed"]), None))
    assert arch["embed"] == c0, "the pre-stack runs at the embedding width"
    k = arch["pre_kernel"]
    for l in range(arch["n_pre"]):
        out.append((f"pre{l}.W", (c0, c0, k), c0 * k))
        out.append((f"pre{l}.b", (c0,), c0 * k))
    for s, u in enumerate(arch["up_rate"]):
        ci, co = arch["channels"][s], arch["channels"][s + 1]
        out.append((f"s{s}.up.W", (ci, co, 2 * u), 2 * ci))
        out.append((f"s{s}.up.b", (co,), 2 * ci))
        for j, kj in enumerate(arch["rb_kernel"]):
            for i, _d in enumerate(arch["dil"]):
                for half in (1, 2):
                    out.append((f"s{s}.rb{j}.d{i}.W{half}", (co, co, kj), co * kj))
                    out.append((f"s{s}.rb{j}.d{i}.b{half}", (co,), co * kj))
    cl = arch["channels"][-1]
    hc = head_channels(arch)
    kh = arch["head_kernel"]
    out.append(("head.W", (hc, cl, kh), cl * kh))
    out.append(("head.b", (hc,), cl * kh))
    nh = arch.get("n_harmonics", 0)
    if nh > 0:
        out.append(("src.merge.W", (nh + 1,), nh + 1))
        out.append(("src.merge.b", (1,), nh + 1))
        out.append(("src.down.W", (cl, 1, arch["hop"]), arch["hop"]))
        out.append(("src.down.b", (cl,), arch["hop"]))
    return out


def blob_floats(arch: dict) -> int:
    return sum(math.prod(shape) for _, shape, _ in tensor_list(arch))


def make_weights(arch: dict, seed: int = 0) -> np.ndarray:
    """The float32 weight blob of `arch` drawn from `seed`."""
    rng = np.random.default_rng(np.random.SeedSequence([seed, 0]))
    parts = []
    for _name, shape, fan_in in tensor_list(arch):
        x = rng.standard_normal(math.prod(shape))
        if fan_in is not None:
            x = x / math.sqrt(fan_in)
        parts.append(x.astype(np.float32))
    return np.concatenate(parts)


def split_weights(arch: dict, blob: np.ndarray) -> dict:
    """Views of the blob by tensor name (for tests that plant special weights)."""
    out, off = {}, 0
    for name, shape, _ in tensor_list(arch):
        n = math.prod(shape)
        out[name] = blob[off:off + n].reshape(shape)
        off += n
    assert off == blob.size
    return out


def make_tokens(arch: dict, batch: int, total_tokens: int, seed: int = 0,
                first_stream: int = 0) -> np.ndarray:
    """int32 [batch][total_tokens] uniform ids; stream b uses SeedSequence([seed, 1, b])."""
    out = np.empty((batch, total_tokens), dtype=np.int32)
    for r in range(batch):
        b = first_stream + r
        rng = np.random.default_rng(np.random.SeedSequence([seed, 1, b]))
        out[r] = rng.integers(0, arch["vocab"], size=total_tokens, dtype=np.int32)
    return out


def frames_per_chunk(arch: dict, tokens: int) -> int:
    """Frames of the pre-stack clock (the f0 clock) in `tokens` tokens."""
    return tokens * arch["frames_per_token"]


def make_f0(arch: dict, batch: int, total_tokens: int, seed: int = 0, first_stream: int = 0) -> np.ndarray:
    """float32 [batch][total_tokens * frames_per_token] fundamental frequency
    per frame (Hz, 0 where unvoiced); stream b uses SeedSequence([seed, 2, b])."""
    F = frames_per_chunk(arch, total_tokens)
    out = np.zeros((batch, F), dtype=np.float32)
    for r in range(batch):
        b = first_stream + r
        rng = np.random.default_rng(np.random.SeedSequence([seed, 2, b]))
        base = rng.uniform(90.0, 250.0)
        walk = 0.0
        f, voiced = 0, bool(rng.integers(0, 2))
        while f < F:
            run = int(rng.geometric(1.0 / (24.0 if voiced else 8.0)))
            for _ in range(min(run, F - f)):
                if voiced:
                    walk += rng.normal(0.0, 0.25)
                    out[r, f] = np.clip(base * 2.0 ** (walk / 12.0), 60.0, 500.0)
                f += 1
            voiced = not voiced
    return out


# ------------------------------------------------------------- flow decoder

def flow_tensor_list(arch: dict):
    """(name, shape, fan_in) for every tensor of the flow decoder's blob, in blob order."""
    D, M, T, H = arch["dim"], arch["n_mel"], arch["t_dim"], arch["mlp"]
    out = [("t.W1", (D, T), T), ("t.b1", (D,), T), ("t.W2", (D, D), D), ("t.b2", (D,), D),
           ("in.W", (D, 4 * M), 4 * M), ("in.b", (D,), 4 * M)]
    for l in range(arch["depth"]):
        out += [(f"b{l}.ada.W", (6 * D, D), D), (f"b{l}.ada.b", (6 * D,), D),
                (f"b{l}.qkv.W", (3 * D, D), D), (f"b{l}.qkv.b", (3 * D,), D),
                (f"b{l}.o.W", (D, D), D), (f"b{l}.o.b", (D,), D),
                (f"b{l}.fc1.W", (H, D), D), (f"b{l}.fc1.b", (H,), D),
                (f"b{l}.fc2.W", (D, H), H), (f"b{l}.fc2.b", (D,), H)]
    out += [("f.ada.W", (2 * D, D), D), ("f.ada.b", (2 * D,), D),
            ("out.W", (M, D), D), ("out.b", (M,), D)]
    return out


def flow_blob_floats(arch: dict) -> int:
    return sum(math.prod(shape) for _, shape, _ in flow_tensor_list(arch))


def make_flow_weights(arch: dict, seed: int = 0) -> np.ndarray:
    """The float32 weight blob of the flow decoder `arch` drawn from `seed`."""
    rng = np.random.default_rng(np.random.SeedSequence([seed, 0]))
    parts = []
    for _name, shape, fan_in in flow_tensor_list(arch):
        parts.append((rng.standard_normal(math.prod(shape)) / math.sqrt(fan_in)).astype(np.float32))
    return np.concatenate(parts)


def split_flow_weights(arch: dict, blob: np.ndarray) -> dict:
    """Views of the flow blob by tensor name."""
    out, off = {}, 0
    for name, shape, _ in flow_tensor_list(arch):
        n = math.prod(shape)
        out[name] = blob[off:off + n].reshape(shape)
        off += n
    assert off == blob.size
    return out


def make_flow_prompt(arch: dict, frames: int, seed: int = 0, stream: int = 0):
    """One turn's prompt of stream `stream`: (mu [frames][n_mel], cond [frames][n_mel],
    spk [n_mel]) float32 from SeedSequence([seed, 4, stream]).  mu and spk are N(0, 1)
    features (the token encoder's output, the speaker embedding); cond stands in for
    the prompt's log-mel spectrogram, N(-5, 2^2)."""
    rng = np.random.default_rng(np.random.SeedSequence([seed, 4, stream]))
    M = arch["n_mel"]
    mu = rng.standard_normal((frames, M)).astype(np.float32)
    cond = (-5.0 + 2.0 * rng.standard_normal((frames, M))).astype(np.float32)
    spk = rng.standard_normal(M).astype(np.float32)
    return mu, cond, spk


def make_flow_mu(arch: dict, batch: int, frames: int, seed: int = 0, first_stream: int = 0) -> np.ndarray:
    """float32 [batch][frames][n_mel] encoder features of the frames after the prompt
    (frame 0 = the first frame of the first chunk), N(0, 1); stream b uses
    SeedSequence([seed, 3, b]).  A call over frames [p, p + n) takes rows p .. p + n - 1,
    so a lookahead frame gets the same features in both calls that present it."""
    out = np.empty((batch, frames, arch["n_mel"]), dtype=np.float32)
    for r in range(batch):
        rng = np.random.default_rng(np.random.SeedSequence([seed, 3, first_stream + r]))
        out[r] = rng.standard_normal((frames, arch["n_mel"]))
    return out
