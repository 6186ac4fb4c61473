"""Oracle for the log-mel front-end (test infrastructure only).

The paper serves Whisper (Section 1; Section 3.1: the encoder consumes fixed
30-s segments).  The front-end is Whisper's: 16 kHz audio, 400-sample frames
with a hop of 160 under a periodic Hann window, the power spectrum of a
400-point DFT (201 bins), a Slaney-style mel filterbank with area
normalisation, log10 with a 1e-10 floor, a dynamic-range clamp 8 below the
clip's maximum and the affine map (x + 4) / 4.

Readings (the paper prints none of this): zero-pad to 480000 samples first,
then reflect-pad 200 on each side (centred frames), keep the first 3000 of
the 3001 frames, take the maximum per clip.

float64 throughout; the DFT is written as its defining sum (a matrix product
with the cos/sin table), not as an FFT.
"""
from __future__ import annotations

import numpy as np

SR = 16000
N_FFT = 400
HOP = 160
N_SAMPLES = 480000
N_FRAMES = 3000


def hann_periodic(n: int = N_FFT) -> np.ndarray:
    i = np.arange(n, dtype=np.float64)
    return 0.5 - 0.5 * np.cos(2.0 * np.pi * i / n)


def frames_of(pcm: np.ndarray) -> np.ndarray:
    """[3000][400] centred frames of a clip zero-padded to 30 s."""
    x = np.zeros(N_SAMPLES, dtype=np.float64)
    n = min(len(pcm), N_SAMPLES)
    x[:n] = pcm[:n]
    xp = np.pad(x, (N_FFT // 2, N_FFT // 2), mode="reflect")   # mirror, edge sample not repeated
    t = np.arange(N_FRAMES)[:, None] * HOP + np.arange(N_FFT)[None, :]
    return xp[t]


def power_spectrum(frames: np.ndarray) -> np.ndarray:
    """|sum_n w[n] x[n] exp(-2 pi i k n / 400)|^2 for k = 0..200."""
    n = np.arange(N_FFT)
    k = np.arange(N_FFT // 2 + 1)
    kn = (k[:, None] * n[None, :]) % N_FFT                      # exact phase index
    ang = 2.0 * np.pi * kn / N_FFT
    xw = frames * hann_periodic()[None, :]
    re = xw @ np.cos(ang).T
    im = -(xw @ np.sin(ang).T)
    return re * re + im * im


def hz_to_mel(f):
    """Slaney mel scale: linear below 1 kHz (3 mel per 200 Hz), logarithmic above."""
    f = np.asarray(f, dtype=np.float64)
    lin = f / (200.0 / 3.0)
    logstep = np.log(6.4) / 27.0
    with np.errstate(divide="ignore"):
        lg = 15.0 + np.log(np.maximum(f, 1e-300) / 1000.0) / logstep
    return np.where(f >= 1000.0, lg, lin)


def mel_to_hz(m):
    m = np.asarray(m, dtype=np.float64)
    lin = m * (200.0 / 3.0)
    logstep = np.log(6.4) / 27.0
    lg = 1000.0 * np.exp(logstep * (m - 15.0))
    return np.where(m >= 15.0, lg, lin)


def mel_filterbank(n_mels: int) -> np.ndarray:
    """[n_mels][201] triangular filters on n_mels+2 mel-spaced edges, area-normalised."""
    fk = np.arange(N_FFT // 2 + 1, dtype=np.float64) * (SR / N_FFT)          # 40 Hz bins
    edges = mel_to_hz(np.linspace(hz_to_mel(0.0), hz_to_mel(SR / 2.0), n_mels + 2))
    W = np.zeros((n_mels, fk.size))
    for m in range(n_mels):
        lo, c, hi = edges[m], edges[m + 1], edges[m + 2]
        rise = (fk - lo) / (c - lo)
        fall = (hi - fk) / (hi - c)
        W[m] = np.maximum(0.0, np.minimum(rise, fall)) * (2.0 / (hi - lo))
    return W


def log_mel(pcm: np.ndarray, n_mels: int) -> np.ndarray:
    """[3000][n_mels] normalised log-mel features of one clip."""
    P = power_spectrum(frames_of(pcm))                       # [3000][201]
    S = P @ mel_filterbank(n_mels).T                         # [3000][n_mels]
    L = np.log10(np.maximum(S, 1e-10))
    L = np.maximum(L, L.max() - 8.0)
    return (L + 4.0) / 4.0
