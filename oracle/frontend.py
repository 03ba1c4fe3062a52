"""Oracle front end: per-segment log-mel features on a 30 s window.

TEST INFRASTRUCTURE ONLY (see oracle/__init__.py).

The paper computes features per chunk, pads or trims them to a 30 s window
and stacks them into a batch (Section 2.3, Listing 1). It names no recipe;
this follows Whisper's published one: 16 kHz audio, 400-sample periodic Hann
window, hop 160, centred frames with reflect padding, power spectrum,
80 or 128 Slaney-normalised mel filters up to 8 kHz, log10 with a 1e-10
floor, clamp to (max - 8), then (x + 4) / 4.

Padding domain: the listing pads the features; the default here pads the
audio with zeros to 30 s before the transform (pad_mode 0), and pad_mode 1
transforms the chunk alone and pads the normalised features with zeros.
"""
import numpy as np

N_FFT = 400
HOP = 160
SR = 16000
N_SAMPLES = 480000  # 30 s
N_FRAMES = 3000     # frames of a 30 s window


def hann_periodic(n: int = N_FFT) -> np.ndarray:
    """w[k] = 0.5 - 0.5 cos(2 pi k / n), k = 0..n-1 (periodic Hann)."""
    k = np.arange(n, dtype=np.float64)
    return 0.5 - 0.5 * np.cos(2.0 * np.pi * k / n)


def frame_audio(x: np.ndarray, n_frames: int) -> np.ndarray:
    """Centred framing: reflect-pad n_fft/2 samples at each end (mirror that
    excludes the edge sample), then frame f covers padded samples
    [hop*f, hop*f + n_fft). Returns [n_frames, n_fft]."""
    x = np.asarray(x, dtype=np.float64)
    xp = np.pad(x, N_FFT // 2, mode="reflect")
    idx = HOP * np.arange(n_frames)[:, None] + np.arange(N_FFT)[None, :]
    return xp[idx]


def power_spectrum(frames: np.ndarray) -> np.ndarray:
    """P[f, k] = |sum_n w[n] x_f[n] exp(-2 pi i k n / N)|^2 for the
    one-sided bins k = 0..N/2. Written as a product with the explicit DFT
    matrix. Returns [n_frames, N/2 + 1]."""
    n = np.arange(N_FFT)
    k = np.arange(N_FFT // 2 + 1)
    dft = np.exp(-2j * np.pi * np.outer(n, k) / N_FFT)  # [N, N/2+1]
    spec = (frames * hann_periodic()[None, :]) @ dft
    return spec.real ** 2 + spec.imag ** 2


def hz_to_mel(f):
    """Slaney mel scale: linear below 1 kHz at 3/200 mel per Hz (1 kHz is
    15 mel), logarithmic above with 27 mel per factor 6.4."""
    f = np.asarray(f, dtype=np.float64)
    lin = 3.0 * f / 200.0
    logstep = np.log(6.4) / 27.0
    with np.errstate(divide="ignore"):
        log = 15.0 + np.log(np.maximum(f, 1e-300) / 1000.0) / logstep
    return np.where(f >= 1000.0, log, lin)


def mel_to_hz(m):
    m = np.asarray(m, dtype=np.float64)
    lin = 200.0 * m / 3.0
    logstep = np.log(6.4) / 27.0
    log = 1000.0 * np.exp(logstep * (m - 15.0))
    return np.where(m >= 15.0, log, lin)


def mel_filterbank(n_mels: int, n_fft: int = N_FFT, sr: int = SR,
                   fmax: float = 8000.0) -> np.ndarray:
    """Slaney-normalised triangular filters on the FFT frequencies.

    n_mels + 2 edge points are equally spaced in mel between mel(0) and
    mel(fmax); filter i rises linearly (in Hz) from edge i to edge i+1 and
    falls to edge i+2, scaled by 2 / (h[i+2] - h[i]). Returns [n_mels,
    n_fft/2 + 1]."""
    fk = np.arange(n_fft // 2 + 1, dtype=np.float64) * sr / n_fft
    h = mel_to_hz(np.linspace(hz_to_mel(0.0), hz_to_mel(fmax), n_mels + 2))
    fb = np.zeros((n_mels, fk.size))
    for i in range(n_mels):
        lower = (fk - h[i]) / (h[i + 1] - h[i])
        upper = (h[i + 2] - fk) / (h[i + 2] - h[i + 1])
        fb[i] = np.maximum(0.0, np.minimum(lower, upper)) * (2.0 / (h[i + 2] - h[i]))
    return fb


def log_mel(x: np.ndarray, n_mels: int, n_frames: int = N_FRAMES) -> np.ndarray:
    """Normalised log-mel of x: frames 0..n_frames-1 of the centred STFT (the
    final centred frame is dropped), mel projection, log10 with floor 1e-10,
    clamp at (max - 8) over the whole window, then (L + 4) / 4.
    Returns [n_mels, n_frames]."""
    p = power_spectrum(frame_audio(x, n_frames))            # [F, 201]
    m = mel_filterbank(n_mels) @ p.T                         # [n_mels, F]
    lg = np.log10(np.maximum(m, 1e-10))
    lg = np.maximum(lg, lg.max() - 8.0)
    return (lg + 4.0) / 4.0


def log_mel_segment(audio: np.ndarray, n_mels: int, pad_mode: int = 0) -> np.ndarray:
    """Features of one segment on the 30 s window, [n_mels, 3000].

    pad_mode 0: zero-pad the audio to 480000 samples, then log_mel.
    pad_mode 1: log_mel of the chunk alone over its n // 160 frames, then pad
    the normalised features with zeros to 3000 frames."""
    a = np.asarray(audio, dtype=np.float64)
    if a.size < 1 or a.size > N_SAMPLES:
        raise ValueError("segment must hold 1..480000 samples")
    if pad_mode == 0:
        return log_mel(np.pad(a, (0, N_SAMPLES - a.size)), n_mels)
    if pad_mode == 1:
        nf = a.size // HOP
        out = np.zeros((n_mels, N_FRAMES))
        if nf > 0:
            out[:, :nf] = log_mel(a, n_mels, nf)
        return out
    raise ValueError("pad_mode must be 0 or 1")
