"""Pins for the log-mel oracle: library DFT, closed forms and special cases.

Fidelity to real Whisper features is parity unpinned: no trained model or
reference features exist here."""
import numpy as np
import pytest

from oracle import mel as M
from paper_2603_11273_amd import synth


def test_shapes():
    for n in (480000, 64000, 1):
        for n_mels in (80, 128):
            assert M.log_mel(np.zeros(n, np.float32) + 0.01, n_mels).shape == (3000, n_mels)
    # 480000 samples, hop 160 -> 3001 centred frames, the last dropped; the stem halves it
    assert 1 + 480000 // 160 - 1 == 3000 and 3000 // 2 == 1500


def test_all_zero_clip_is_constant():
    """Silence: every power is 0 -> log10 floor -10 -> (-10 + 4) / 4 = -1.5 exactly."""
    out = M.log_mel(np.zeros(16000, np.float32), 80)
    assert np.all(out == -1.5)


def test_framing_reflect_pad():
    x = np.arange(1, 1001, dtype=np.float64)
    fr = M.frames_of(x)
    # frame 0 is centred on sample 0: x[200], ..., x[1], x[0], x[1], ..., x[199]
    expect0 = np.array([x[abs(n - 200)] for n in range(400)])
    assert np.array_equal(fr[0], expect0)
    # frame 3 starts at sample 3*160 - 200
    assert np.array_equal(fr[3], x[280:680])
    # frames past the audio read the zero padding
    assert np.all(fr[100] == 0.0)


def test_dft_matches_fft():
    rng = np.random.default_rng(0)
    frames = rng.standard_normal((7, 400))
    P = M.power_spectrum(frames)
    ref = np.abs(np.fft.rfft(frames * np.hanning(401)[:400], n=400)) ** 2
    # np.hanning(401)[:400] is the periodic Hann window of length 400
    assert np.allclose(P, ref, rtol=1e-10, atol=1e-9)


def test_tone_peaks_at_its_bin():
    t = np.arange(480000) / 16000.0
    x = np.sin(2 * np.pi * 1000.0 * t)
    P = M.power_spectrum(M.frames_of(x)[1000:1003])
    assert np.all(np.argmax(P, axis=1) == 25)                 # 1000 Hz / 40 Hz per bin


def test_mel_scale_closed_forms():
    assert M.hz_to_mel(1000.0) == pytest.approx(15.0, abs=1e-12)
    assert M.hz_to_mel(200.0) == pytest.approx(3.0, abs=1e-12)
    assert M.hz_to_mel(6400.0) == pytest.approx(42.0, abs=1e-12)   # 15 + 27
    f = np.linspace(0, 8000, 97)
    assert np.allclose(M.mel_to_hz(M.hz_to_mel(f)), f, atol=1e-9)


@pytest.mark.parametrize("n_mels", [80, 128])
def test_filterbank_partition_of_unity(n_mels):
    W = M.mel_filterbank(n_mels)
    assert W.shape == (n_mels, 201) and np.all(W >= 0)
    edges = M.mel_to_hz(np.linspace(M.hz_to_mel(0.0), M.hz_to_mel(8000.0), n_mels + 2))
    # undo the area normalisation: the triangles then sum to 1 between the
    # first and the last centre frequency
    tri = W * ((edges[2:] - edges[:-2]) / 2.0)[:, None]
    fk = np.arange(201) * 40.0
    inside = (fk >= edges[1]) & (fk <= edges[n_mels])
    assert np.allclose(tri.sum(axis=0)[inside], 1.0, atol=1e-12)
    # each triangle peaks at 1 on its centre and is 0 at its two edges
    assert np.all(tri.max(axis=1) <= 1.0 + 1e-12)


def test_dynamic_range_clamp():
    pcm = synth.pcm_clip(1, 0, 64000)
    out = M.log_mel(pcm, 80)
    top = out.max()
    assert np.isclose(out.min(), top - 2.0)                    # (m - 8 + 4)/4 = top - 2
    assert out[-1].max() == pytest.approx(top - 2.0)          # padded frames sit on the clamp
