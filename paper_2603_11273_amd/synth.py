"""Seeded synthetic inputs for the batched Whisper-shaped ASR step.

This module is shared by the oracle tests, the GPU parity tests and the
benchmark.  It holds none of the method's arithmetic: it only draws data with
the shapes and distributions of the paper's workloads (Section 4, setup:
LibriSpeech-like right-skewed durations, a flat synthetic duration split,
Poisson arrivals) and the Whisper-shaped model sizes the build is measured on.

Two kinds of generator live here.

* Small host-side data (PCM clips, durations, arrival times, token ids) comes
  from numpy's seeded PCG64 generator.
* Large tensors (model parameters, synthetic encoder outputs, pre-filled
  self-attention caches) come from a counter-based integer hash so the very
  same values can be produced on the CPU (for the oracle, with torch integer
  ops) and directly in device memory (for the benchmark at full size, with
  the small HIP kernel of libasr_synth.so) without a multi-gigabyte host
  round trip.  The hash is Chris Wellons' "lowbias32" integer mixer
  (published with his hash-prospector project); every value it yields is an
  integer multiple of a power of two with at most 8 significant bits, so it
  is exactly representable in float32 *and* bfloat16.  That makes the
  bf16-path inputs identical on both sides with no rounding step.  The
  "fine" variant adds a second draw 2^10 times finer (at most 18
  significant bits: exact in float32, generally not in bfloat16), for the
  parity cases that must see weights the bf16 path has to round.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field

import numpy as np

SAMPLE_RATE = 16000
N_SAMPLES_30S = 480000          # 30 s at 16 kHz: one encoder segment (Section 3.1)
N_AUDIO_CTX = 1500              # encoder positions per 30-s segment
N_TEXT_CTX = 448                # maximum output tokens (Section 4.1, setup)

_M32 = 0xFFFFFFFF


# ----------------------------------------------------------------------------
# Model shapes (Whisper family sizes; weights are random, never trained)
# ----------------------------------------------------------------------------
@dataclass(frozen=True)
class ModelShape:
    name: str
    n_mels: int
    d_model: int
    n_enc: int
    n_dec: int
    n_head: int
    d_ffn: int
    vocab: int
    dtype: str                  # "f32" or "bf16": storage type of matrices/activations

    @property
    def d_head(self) -> int:
        return self.d_model // self.n_head


SHAPES = {
    "tiny": ModelShape("tiny", 80, 384, 4, 4, 6, 1536, 51865, "f32"),
    "base": ModelShape("base", 80, 512, 6, 6, 8, 2048, 51865, "bf16"),
    "small": ModelShape("small", 80, 768, 12, 12, 12, 3072, 51865, "bf16"),
    "large-v3": ModelShape("large-v3", 128, 1280, 32, 32, 20, 5120, 51866, "bf16"),
}


def reduced_shape(shape: ModelShape, n_enc: int, n_dec: int, vocab: int | None = None,
                  dtype: str | None = None) -> ModelShape:
    """Same widths, fewer layers / smaller vocabulary: for fast parity cases."""
    return ModelShape(shape.name + f"-l{n_enc}x{n_dec}", shape.n_mels, shape.d_model, n_enc,
                      n_dec, shape.n_head, shape.d_ffn, vocab or shape.vocab,
                      dtype or shape.dtype)


@dataclass(frozen=True)
class Workload:
    name: str
    shape: str
    seed: int
    batch: int
    note: str
    extra: dict = field(default_factory=dict)


# The five measured workloads.  Seeds are 20260311 + index.
WORKLOADS = {
    "tiny-fp32": Workload("tiny-fp32", "tiny", 20260311, 1,
                          "one 4-s clip, 16 teacher-forced steps", {"clip_s": 4.0, "steps": 16}),
    "base-bf16": Workload("base-bf16", "base", 20260312, 8,
                          "lognormal durations (median 6 s, sigma 0.6) clipped to [1,30] s"),
    "small-bf16-hrrn": Workload("small-bf16-hrrn", "small", 20260313, 32,
                                "256 Poisson requests (20/s), durations U[1,30] s, HRRN batches of 32",
                                {"n_requests": 256, "rate": 20.0}),
    "large-v3-encoder": Workload("large-v3-encoder", "large-v3", 20260314, 64,
                                 "64 full 30-s clips through the encoder"),
    "large-v3-decode": Workload("large-v3-decode", "large-v3", 20260315, 128,
                                "128 sequences, self-KV lengths U[10,400], 1500 cross positions",
                                {"n_requests": 2000, "kv_lo": 10, "kv_hi": 400}),
}


# ----------------------------------------------------------------------------
# Counter-based hash generator (bit-identical on CPU and GPU)
# ----------------------------------------------------------------------------
def lowbias32_py(x: int) -> int:
    """Chris Wellons' lowbias32 mixer on a Python int (reference definition)."""
    x &= _M32
    x ^= x >> 16
    x = (x * 0x7FEB352D) & _M32
    x ^= x >> 15
    x = (x * 0x846CA68B) & _M32
    x ^= x >> 16
    return x


def stream_keys(seed: int, stream: int) -> tuple[int, int]:
    k1 = lowbias32_py((seed & _M32) ^ lowbias32_py(stream & _M32))
    k2 = lowbias32_py(k1 ^ 0x5BD1E995)
    return k1, k2


def hash_py(seed: int, stream: int, idx: int) -> int:
    k1, k2 = stream_keys(seed, stream)
    return lowbias32_py((lowbias32_py(idx ^ k1) + k2) & _M32)


def _mul32_t(x, c: int):
    # (x * c) mod 2^32 for int64 tensors holding values < 2^32, with no
    # intermediate above 2^49 (so no signed overflow anywhere).
    lo, hi = c & 0xFFFF, c >> 16
    return (x * lo + (((x * hi) & 0xFFFF) << 16)) & _M32


def _lowbias32_t(x):
    x = x ^ (x >> 16)
    x = _mul32_t(x, 0x7FEB352D)
    x = x ^ (x >> 15)
    x = _mul32_t(x, 0x846CA68B)
    x = x ^ (x >> 16)
    return x


def hash_tensor(seed: int, stream: int, start: int, count: int, device="cpu"):
    """uint32 hash values (in int64) for counters start .. start+count-1."""
    import torch
    k1, k2 = stream_keys(seed, stream)
    idx = torch.arange(start, start + count, dtype=torch.int64, device=device)
    h = _lowbias32_t(idx ^ k1)
    return _lowbias32_t((h + k2) & _M32)


FINE_STREAM = 0x80000000          # stream id offset of the fine term's draws

_SYNTH_LIB = None


def _synth_lib():
    """The device generator (libasr_synth.so, built next to this file)."""
    global _SYNTH_LIB
    if _SYNTH_LIB is None:
        import ctypes as C
        import os

        import torch  # noqa: F401  (binds the library to torch's HIP runtime)
        path = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libasr_synth.so")
        if not os.path.exists(path):
            raise ImportError(f"{path} is missing: build it with "
                              "`python -m paper_2603_11273_amd.build`")
        lib = C.CDLL(path)
        lib.asr_synth_grid.restype = C.c_int
        lib.asr_synth_grid.argtypes = [C.c_void_p, C.c_int64, C.c_uint32, C.c_uint32, C.c_uint32,
                                       C.c_int32, C.c_int32, C.c_float, C.c_int32, C.c_uint32,
                                       C.c_uint32, C.c_void_p]
        _SYNTH_LIB = lib
    return _SYNTH_LIB


def grid_values(seed: int, stream: int, shape, kmax: int, bits: int, device="cpu",
                offset: float = 0.0, chunk: int = 1 << 24, fine: bool = False):
    """float32 tensor of (k * 2^-bits + offset), k uniform on [-kmax, kmax].

    kmax <= 255 keeps every k*2^-bits exactly representable in bfloat16; with
    offset 1.0 (LayerNorm gains) the value is still exact in float32.  fine:
    plus j * 2^-(bits + 10), j uniform on [-255, 255] from the stream
    FINE_STREAM + stream (exact in float32, generally not in bfloat16).
    CPU tensors come from torch integer ops, device tensors from the HIP
    generator; the two agree bit for bit.
    """
    import torch
    assert 0 < kmax <= 255
    numel = int(np.prod(shape)) if len(shape) else 1
    assert numel <= 1 << 32
    out = torch.empty(numel, dtype=torch.float32, device=device)
    if out.device.type != "cpu":
        k1, k2 = stream_keys(seed, stream)
        f1, f2 = stream_keys(seed, FINE_STREAM + stream)
        with torch.cuda.device(out.device):
            st = torch.cuda.current_stream().cuda_stream
            rc = _synth_lib().asr_synth_grid(out.data_ptr(), numel, 0, k1, k2, kmax, bits,
                                             float(offset), int(fine), f1, f2, st)
        if rc != 0:
            raise RuntimeError(f"asr_synth_grid failed ({rc})")
        return out.view(*shape)
    levels = 2 * kmax + 1
    scale = 2.0 ** (-bits)
    for s in range(0, numel, chunk):
        n = min(chunk, numel - s)
        h = hash_tensor(seed, stream, s, n, device)
        k = ((h * levels) >> 32) - kmax
        v = k.to(torch.float32) * scale
        if offset:
            v = v + offset
        if fine:
            j = ((hash_tensor(seed, FINE_STREAM + stream, s, n, device) * 511) >> 32) - 255
            v = v + j.to(torch.float32) * 2.0 ** (-(bits + 10))
        out[s:s + n] = v
    return out.view(*shape)


# ----------------------------------------------------------------------------
# Model parameters
# ----------------------------------------------------------------------------
def param_specs(shape: ModelShape):
    """Ordered (name, shape, kind) for every parameter tensor.

    kind: "w" matrix/bias ~ std 0.02, "g" LayerNorm gain 1 + small, "b"
    LayerNorm shift.  The order is the load order of the C ABI.
    """
    d, f, m = shape.d_model, shape.d_ffn, shape.n_mels
    specs = []
    if shape.n_enc > 0:
        specs += [("conv1.w", (d, m, 3), "w"), ("conv1.b", (d,), "w"),
                  ("conv2.w", (d, d, 3), "w"), ("conv2.b", (d,), "w")]
        for l in range(shape.n_enc):
            p = f"enc.{l}."
            specs += [(p + "attn_ln.g", (d,), "g"), (p + "attn_ln.b", (d,), "b"),
                      (p + "q.w", (d, d), "w"), (p + "q.b", (d,), "w"),
                      (p + "k.w", (d, d), "w"),
                      (p + "v.w", (d, d), "w"), (p + "v.b", (d,), "w"),
                      (p + "o.w", (d, d), "w"), (p + "o.b", (d,), "w"),
                      (p + "mlp_ln.g", (d,), "g"), (p + "mlp_ln.b", (d,), "b"),
                      (p + "fc1.w", (f, d), "w"), (p + "fc1.b", (f,), "w"),
                      (p + "fc2.w", (d, f), "w"), (p + "fc2.b", (d,), "w")]
        specs += [("ln_post.g", (d,), "g"), ("ln_post.b", (d,), "b")]
    if shape.n_dec > 0:
        specs += [("tok_emb", (shape.vocab, d), "w"), ("pos_emb", (N_TEXT_CTX, d), "w")]
        for l in range(shape.n_dec):
            p = f"dec.{l}."
            specs += [(p + "attn_ln.g", (d,), "g"), (p + "attn_ln.b", (d,), "b"),
                      (p + "q.w", (d, d), "w"), (p + "q.b", (d,), "w"),
                      (p + "k.w", (d, d), "w"),
                      (p + "v.w", (d, d), "w"), (p + "v.b", (d,), "w"),
                      (p + "o.w", (d, d), "w"), (p + "o.b", (d,), "w"),
                      (p + "xattn_ln.g", (d,), "g"), (p + "xattn_ln.b", (d,), "b"),
                      (p + "xq.w", (d, d), "w"), (p + "xq.b", (d,), "w"),
                      (p + "xk.w", (d, d), "w"),
                      (p + "xv.w", (d, d), "w"), (p + "xv.b", (d,), "w"),
                      (p + "xo.w", (d, d), "w"), (p + "xo.b", (d,), "w"),
                      (p + "mlp_ln.g", (d,), "g"), (p + "mlp_ln.b", (d,), "b"),
                      (p + "fc1.w", (f, d), "w"), (p + "fc1.b", (f,), "w"),
                      (p + "fc2.w", (d, f), "w"), (p + "fc2.b", (d,), "w")]
        specs += [("ln.g", (d,), "g"), ("ln.b", (d,), "b")]
    return specs


def model_params(shape: ModelShape, seed: int, device="cpu", fine: bool = False):
    """Ordered dict name -> float32 tensor.  Values are exact in bfloat16,
    unless fine (then every tensor carries the finer second draw)."""
    params = {}
    for i, (name, shp, kind) in enumerate(param_specs(shape)):
        if kind == "g":
            params[name] = grid_values(seed, i, shp, 141, 12, device, offset=1.0, fine=fine)
        else:
            params[name] = grid_values(seed, i, shp, 141, 12, device, fine=fine)
    return params


def bf16_rounded_params(params: dict) -> dict:
    """The parameters as a bf16 context holds them: matrices (linear and conv
    weights, the token embedding) rounded to bfloat16 (round to nearest
    even, torch's conversion) and back to float32; vectors (biases, LayerNorm
    gains and shifts, positional embeddings) stay float32."""
    import torch
    out = {}
    for name, t in params.items():
        if name.endswith(".w") or name == "tok_emb":
            out[name] = t.to(torch.bfloat16).to(torch.float32)
        else:
            out[name] = t
    return out


def encoder_output(seed: int, index: int, d_model: int, device="cpu"):
    """Synthetic encoder output E [1500][d], std ~1, bf16-exact (stream 10^6 + index)."""
    return grid_values(seed, 1_000_000 + index, (N_AUDIO_CTX, d_model), 221, 7, device)


def self_kv_prefix(seed: int, index: int, n_layers: int, n_head: int, d_head: int = 64,
                   device="cpu"):
    """Synthetic self-attention cache [L][2][H][448][64], std ~0.7; a sequence
    with a pre-filled length L uses positions [0, L)."""
    return grid_values(seed, 2_000_000 + index, (n_layers, 2, n_head, N_TEXT_CTX, d_head), 155,
                       7, device)


# ----------------------------------------------------------------------------
# Host-side workload data
# ----------------------------------------------------------------------------
def pcm_clip(seed: int, index: int, n_samples: int) -> np.ndarray:
    """Sum of 3 sines plus N(0, 0.05) noise, float32, `n_samples` long.

    f ~ U[100, 4000] Hz, amplitude ~ U[0.1, 0.3], phase ~ U[0, 2 pi).
    """
    rng = np.random.default_rng([seed, 7, index])
    f = rng.uniform(100.0, 4000.0, 3)
    a = rng.uniform(0.1, 0.3, 3)
    ph = rng.uniform(0.0, 2.0 * np.pi, 3)
    t = np.arange(n_samples, dtype=np.float64) / SAMPLE_RATE
    x = np.zeros(n_samples, dtype=np.float64)
    for i in range(3):
        x += a[i] * np.sin(2.0 * np.pi * f[i] * t + ph[i])
    x += rng.normal(0.0, 0.05, n_samples)
    return x.astype(np.float32)


def durations_lognormal(seed: int, n: int, median_s: float = 6.0, sigma: float = 0.6,
                        lo: float = 1.0, hi: float = 30.0) -> np.ndarray:
    """Right-skewed durations standing in for LibriSpeech test-clean (Section 4.1)."""
    rng = np.random.default_rng([seed, 11])
    d = np.exp(math.log(median_s) + sigma * rng.standard_normal(n))
    return np.clip(d, lo, hi)


def durations_uniform(seed: int, n: int, lo: float = 1.0, hi: float = 30.0) -> np.ndarray:
    """Flat durations standing in for the synthetic split (Section 4.1)."""
    rng = np.random.default_rng([seed, 13])
    return rng.uniform(lo, hi, n)


def n_samples_of(durations_s) -> np.ndarray:
    return np.rint(np.asarray(durations_s) * SAMPLE_RATE).astype(np.int64)


def poisson_arrivals_us(seed: int, n: int, rate_per_s: float) -> np.ndarray:
    """Poisson arrival times (burstiness 1.0) in integer microseconds."""
    rng = np.random.default_rng([seed, 17])
    gaps = rng.exponential(1.0 / rate_per_s, n)
    return np.rint(np.cumsum(gaps) * 1e6).astype(np.int64)


def token_ids(seed: int, shape, vocab: int) -> np.ndarray:
    rng = np.random.default_rng([seed, 19])
    return rng.integers(0, vocab, size=shape, dtype=np.int64).astype(np.int32)


def kv_lengths(seed: int, n: int, lo: int = 10, hi: int = 400) -> np.ndarray:
    rng = np.random.default_rng([seed, 23])
    return rng.integers(lo, hi + 1, size=n, dtype=np.int64).astype(np.int32)


ATTENTION_CASES = ("small", "first_tile_large", "late_large", "late_huge", "very_negative")


def attention_operands(seed: int, n: int, d_model: int, case: str):
    """q, k, v [n][1500][d] float32 for the encoder attention kernel, every
    value bf16-exact (sixteenths in [-1/4, 1/4], plus +-1 components).

    Each head's queries and keys are small random parts plus, depending on
    `case`, a shared +-1 pattern u per head (|u|^2 = 64): 'small' has none;
    'first_tile_large' adds u to the queries and 1.5 u to keys 0..63;
    'late_large' adds u to the queries and 1.5 u to keys 900..963;
    'late_huge' adds u to the queries and 2.5 u to keys 900..963;
    'very_negative' adds u to the queries and -1.5 u to every key.  With q
    read in the exp2 domain, the structured keys score about +-96 (+160 for
    'late_huge', past the 2^128 range of exp2 in fp32 against a reference
    of 0; the rest stay within a few units), which moves the kernel's
    softmax reference."""
    assert case in ATTENTION_CASES
    rng = np.random.default_rng([seed, 29, ATTENTION_CASES.index(case)])
    shp = (n, N_AUDIO_CTX, d_model)
    q = rng.integers(-4, 5, size=shp).astype(np.float32) / 16
    k = rng.integers(-4, 5, size=shp).astype(np.float32) / 16
    v = rng.integers(-8, 9, size=shp).astype(np.float32) / 8
    u = rng.choice(np.array([-1.0, 1.0], np.float32), size=(1, 1, d_model))
    if case != "small":
        q += u
        if case == "first_tile_large":
            k[:, 0:64] += 1.5 * u
        elif case == "late_large":
            k[:, 900:964] += 1.5 * u
        elif case == "late_huge":
            k[:, 900:964] += 2.5 * u
        else:
            k += -1.5 * u
    return q, k, v
