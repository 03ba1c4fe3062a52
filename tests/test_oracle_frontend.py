"""Pins for the oracle's log-mel front end (padding, framing, Hann window,
power spectrum, Slaney mel filter bank, log and normalisation).

Each check compares against something other than the oracle itself: the
FFT library, closed forms of the DFT of a windowed tone, Parseval's
identity, the Slaney mel scale's defining values, and an independent
library implementation of the same recipe (transformers' audio utilities
and Whisper feature extractor, CPU)."""
import numpy as np
import pytest

import oracle
from oracle import frontend as F


def _rng(seed=0):
    return np.random.Generator(np.random.PCG64(seed))


def test_power_spectrum_matches_fft_library():
    x = _rng(1).standard_normal((7, 400))
    want = np.abs(np.fft.rfft(x * np.hanning(401)[:-1], axis=-1)) ** 2
    got = F.power_spectrum(x)
    assert np.allclose(got, want, rtol=1e-11, atol=1e-9)


def test_hann_is_periodic_hann():
    w = F.hann_periodic(400)
    # periodic Hann of length N is the symmetric Hann of length N+1 minus its last point
    assert np.allclose(w, np.hanning(401)[:-1], atol=1e-15)
    assert w[0] == 0.0 and abs(w[200] - 1.0) < 1e-15


def test_parseval_one_sided():
    x = _rng(2).standard_normal((5, 400))
    p = F.power_spectrum(x)
    y = x * F.hann_periodic()[None]
    one_sided = p[:, 0] + 2 * p[:, 1:200].sum(1) + p[:, 200]
    assert np.allclose(one_sided, 400 * (y ** 2).sum(1), rtol=1e-11)


@pytest.mark.parametrize("k0", [11, 25, 75, 150])
def test_tone_at_bin_centre_closed_form(k0):
    # x[n] = cos(2 pi k0 n / N + phi) under a periodic Hann window: |X_k0| = N/4,
    # |X_{k0+-1}| = N/8, zero elsewhere, whatever the phase.
    n = np.arange(480000)
    x = np.cos(2 * np.pi * (40.0 * k0) * n / 16000 + 0.3)
    p = F.power_spectrum(F.frame_audio(x, 3000))[5:-5]      # interior frames
    assert np.allclose(p[:, k0], 1e4, rtol=1e-9)
    assert np.allclose(p[:, k0 - 1], 2500, rtol=1e-9)
    assert np.allclose(p[:, k0 + 1], 2500, rtol=1e-9)
    rest = np.delete(p, [k0 - 1, k0, k0 + 1], axis=1)
    assert rest.max() < 1e-12 * 1e4


def test_frame_reflect_padding():
    x = np.arange(1000, dtype=np.float64)
    fr = F.frame_audio(x, 4)
    # frame 0 covers padded samples 0..399 = x[200], x[199], ..., x[1], x[0], ..., x[199]
    assert np.array_equal(fr[0, :200], x[200:0:-1])
    assert np.array_equal(fr[0, 200:], x[:200])
    assert np.array_equal(fr[1], np.concatenate([x[40:0:-1], x[:360]]))
    assert np.array_equal(fr[2], x[120:520])


def test_slaney_mel_scale_defining_values():
    assert F.hz_to_mel(1000.0) == pytest.approx(15.0, abs=1e-12)
    assert F.hz_to_mel(500.0) == pytest.approx(7.5, abs=1e-12)
    assert F.hz_to_mel(6400.0) == pytest.approx(42.0, abs=1e-12)    # one factor 6.4 = 27 mel
    f = np.array([0.0, 123.0, 999.0, 1000.0, 1001.0, 4321.0, 8000.0])
    assert np.allclose(F.mel_to_hz(F.hz_to_mel(f)), f, rtol=1e-13, atol=1e-10)


@pytest.mark.parametrize("n_mels", [80, 128])
def test_filterbank_matches_library(n_mels):
    au = pytest.importorskip("transformers.audio_utils")
    lib = au.mel_filter_bank(num_frequency_bins=201, num_mel_filters=n_mels, min_frequency=0.0,
                             max_frequency=8000.0, sampling_rate=16000, norm="slaney",
                             mel_scale="slaney")
    assert np.allclose(F.mel_filterbank(n_mels), lib.T, rtol=1e-10, atol=1e-13)


@pytest.mark.parametrize("n_mels", [80, 128])
def test_filterbank_unit_area(n_mels):
    # Slaney normalisation gives every triangle unit area in Hz; the Riemann
    # sum over 40 Hz bins approaches 1 for filters much wider than a bin.
    fb = F.mel_filterbank(n_mels)
    h = F.mel_to_hz(np.linspace(0.0, F.hz_to_mel(8000.0), n_mels + 2))
    wide = (h[2:] - h[:-2]) > 300.0
    assert wide.sum() >= 8
    assert np.allclose(fb[wide].sum(1) * 40.0, 1.0, atol=0.012)


@pytest.mark.parametrize("n_mels", [80, 128])
def test_log_mel_matches_library(n_mels):
    tf = pytest.importorskip("transformers")
    from paper_2507_01021_amd import synth
    audio = synth.synth_audio(_rng(3), 112000)
    fe = tf.WhisperFeatureExtractor(feature_size=n_mels)
    lib = fe(audio, sampling_rate=16000, return_tensors="np").input_features[0]
    got = F.log_mel_segment(audio, n_mels, 0)
    assert got.shape == (n_mels, 3000)
    assert np.abs(got - lib).max() < 2e-5    # the library works in float32


@pytest.mark.parametrize("n_mels,f0", [(80, 440.0), (80, 1000.0), (80, 3000.0),
                                         (128, 440.0), (128, 1000.0), (128, 3000.0)])
def test_tone_peak_mel_bin_and_value(n_mels, f0):
    # A unit tone at FFT bin centre k0 = f0 / 40 has interior power 1e4 at k0
    # and 2500 at k0 +- 1, so the mel value of filter i is
    # 1e4 fb[i,k0] + 2500 (fb[i,k0-1] + fb[i,k0+1]); the peak is the filter
    # whose centre lies nearest the tone.
    k0 = int(f0 / 40)
    n = np.arange(480000)
    x = np.sin(2 * np.pi * f0 * n / 16000)
    y = F.log_mel(x, n_mels)
    fb = F.mel_filterbank(n_mels)
    m = 1e4 * fb[:, k0] + 2500 * (fb[:, k0 - 1] + fb[:, k0 + 1])
    peak = int(np.argmax(m))
    h = F.mel_to_hz(np.linspace(0.0, F.hz_to_mel(8000.0), n_mels + 2))
    nearest = int(np.argmin(np.abs(h[1:-1] - f0)))
    assert abs(peak - nearest) <= 1
    mid = y[:, 10:-10]
    assert np.all(np.argmax(mid, axis=0) == peak)
    assert np.allclose(mid[peak], (np.log10(m[peak]) + 4) / 4, atol=1e-9)
    # every value sits at or above the floor max - 8 (in log10 units)
    assert y.min() >= y.max() - 2.0 - 1e-12


def test_normalisation_range_and_floor():
    from paper_2507_01021_amd import synth
    a = synth.synth_audio(_rng(4), 48000)
    y = F.log_mel_segment(a, 80, 0)
    # zero-padded frames have zero power: floor 1e-10 then clamp to max - 8
    assert y.max() - y.min() == pytest.approx(2.0, abs=1e-12)
    assert np.allclose(y[:, 400:], y.max() - 2.0, atol=1e-12)


def test_pad_mode_feature_domain():
    from paper_2507_01021_amd import synth
    a = synth.synth_audio(_rng(5), 48123)
    y = F.log_mel_segment(a, 80, 1)
    nf = 48123 // 160
    assert np.all(y[:, nf:] == 0.0)
    assert np.allclose(y[:, :nf], F.log_mel(a, 80, nf))
    assert y[:, :nf].max() - y[:, :nf].min() <= 2.0 + 1e-12


def test_segment_length_validation():
    with pytest.raises(ValueError):
        F.log_mel_segment(np.zeros(0), 80)
    with pytest.raises(ValueError):
        F.log_mel_segment(np.zeros(480001), 80)
    assert oracle.log_mel_segment(np.zeros(480000) + 0.1, 80).shape == (80, 3000)
