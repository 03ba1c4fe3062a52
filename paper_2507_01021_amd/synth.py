"""Seeded synthetic inputs: model shapes, random weights, audio segments and
multi-user workloads.

This module is the only code shared by the CPU oracle and the GPU path. It
holds none of the model's arithmetic: it draws numbers, fixes shapes and
packs bytes.

* Weights follow the paper's setting of fine-tuned Whisper checkpoints
  (Section 2, "Approach"); none ship here, so every tensor is drawn from
  N(0, 0.02) with a fixed seed, layer-norm gains as 1 + N(0, 0.02).
  Half-precision models round each fp32 draw to bfloat16 (nearest-even).
* Segments follow the paper's VAD output of 3-30 s speech pieces
  (Section 2.1): 16 kHz mono audio, a sum of three sinusoids plus Gaussian
  noise, one segment per independent unit (Section 2.3).
* Multi-user workloads follow the central priority queue of Section 2.2:
  each simulated user emits segments with exponential inter-arrival times.
"""
from __future__ import annotations

import dataclasses
import struct
from concurrent.futures import ThreadPoolExecutor

import numpy as np

SAMPLE_RATE = 16000
N_SAMPLES_30S = 480000  # 30 s window at 16 kHz
N_AUDIO_CTX = 1500
N_TEXT_CTX = 448


@dataclasses.dataclass(frozen=True)
class ModelShape:
    name: str
    n_mels: int
    d: int
    n_head: int
    n_enc: int
    n_dec: int
    n_vocab: int
    dtype: str  # "f32" or "bf16"
    n_audio_ctx: int = N_AUDIO_CTX
    n_text_ctx: int = N_TEXT_CTX

    @property
    def head_dim(self) -> int:
        return self.d // self.n_head

    def with_(self, **kw) -> "ModelShape":
        return dataclasses.replace(self, **kw)


# Whisper-family shapes used by the workloads (head dim 64 in all of them).
TINY = ModelShape("tiny", 80, 384, 6, 4, 4, 51865, "f32")
BASE = ModelShape("base", 80, 512, 8, 6, 6, 51865, "bf16")
SMALL = ModelShape("small", 80, 768, 12, 12, 12, 51865, "bf16")
LARGE_V3 = ModelShape("large-v3", 128, 1280, 20, 32, 32, 51866, "bf16")
TURBO = ModelShape("large-v3-turbo", 128, 1280, 20, 32, 4, 51866, "bf16")
# Encoder-only CTC models (n_dec = 0): the encoder of the named shape and a
# linear head to n_vocab ids, id 0 the blank.
CTC_TINY = ModelShape("ctc-tiny", 80, 384, 6, 4, 0, 256, "f32")
CTC_BASE = ModelShape("ctc-base", 80, 512, 8, 6, 0, 1024, "bf16")
SHAPES = {s.name: s for s in (TINY, BASE, SMALL, LARGE_V3, TURBO, CTC_TINY, CTC_BASE)}


def prompt_for(shape: ModelShape) -> list[int]:
    """Start-of-transcript, language, task and no-timestamps ids (the prompt
    plus no-timestamp token of Section 2.3). With random weights only their
    range matters; both sides receive the same list."""
    if shape.n_dec == 0:
        return []  # CTC models take no prompt
    if shape.n_vocab >= 51866:
        return [50258, 50259, 50360, 50364]
    return [50258, 50259, 50359, 50363]


# ----------------------------------------------------------------------------
# weights
# ----------------------------------------------------------------------------

def _attn_specs(prefix: str, d: int):
    return [
        (prefix + ".q.w", (d, d), "w"), (prefix + ".q.b", (d,), "w"),
        (prefix + ".k.w", (d, d), "w"),
        (prefix + ".v.w", (d, d), "w"), (prefix + ".v.b", (d,), "w"),
        (prefix + ".o.w", (d, d), "w"), (prefix + ".o.b", (d,), "w"),
    ]


def _ln_specs(prefix: str, d: int):
    return [(prefix + ".g", (d,), "g"), (prefix + ".b", (d,), "w")]


def _mlp_specs(prefix: str, d: int):
    return [
        (prefix + ".fc1.w", (4 * d, d), "w"), (prefix + ".fc1.b", (4 * d,), "w"),
        (prefix + ".fc2.w", (d, 4 * d), "w"), (prefix + ".fc2.b", (d,), "w"),
    ]


def tensor_specs(shape: ModelShape):
    """Canonical tensor order (name, shape, kind). Matrices are [out, in];
    conv kernels are [out, in, tap]. This order is also the weight-blob order
    documented in the C header."""
    d = shape.d
    specs = [
        ("enc.conv1.w", (d, shape.n_mels, 3), "w"), ("enc.conv1.b", (d,), "w"),
        ("enc.conv2.w", (d, d, 3), "w"), ("enc.conv2.b", (d,), "w"),
    ]
    for i in range(shape.n_enc):
        p = f"enc.{i}"
        specs += _ln_specs(p + ".attn_ln", d) + _attn_specs(p + ".attn", d)
        specs += _ln_specs(p + ".mlp_ln", d) + _mlp_specs(p + ".mlp", d)
    specs += _ln_specs("enc.ln_post", d)
    if shape.n_dec == 0:  # encoder-only CTC model: the head instead of a decoder
        return specs + [("ctc.w", (shape.n_vocab, d), "w"), ("ctc.b", (shape.n_vocab,), "w")]
    specs += [("dec.tok_emb", (shape.n_vocab, d), "w"),
              ("dec.pos_emb", (shape.n_text_ctx, d), "w")]
    for i in range(shape.n_dec):
        p = f"dec.{i}"
        specs += _ln_specs(p + ".attn_ln", d) + _attn_specs(p + ".attn", d)
        specs += _ln_specs(p + ".cross_ln", d) + _attn_specs(p + ".cross", d)
        specs += _ln_specs(p + ".mlp_ln", d) + _mlp_specs(p + ".mlp", d)
    specs += _ln_specs("dec.ln", d)
    return specs


def round_to_bf16(a: np.ndarray) -> np.ndarray:
    """fp32 -> bf16 bit patterns (uint16), round to nearest even (no NaNs
    occur in the drawn values)."""
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32)
    r = (u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))) >> np.uint32(16)
    return r.astype(np.uint16)


def bf16_to_f32(b: np.ndarray) -> np.ndarray:
    return (b.astype(np.uint32) << np.uint32(16)).view(np.float32)


def _draw(seed: int, index: int, shp, kind: str, dtype: str):
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, index])))
    a = rng.standard_normal(int(np.prod(shp)), dtype=np.float32)
    a *= np.float32(0.02)
    if kind == "g":
        a += np.float32(1.0)
    a = a.reshape(shp)
    if dtype == "bf16":
        bits = round_to_bf16(a)
        return bf16_to_f32(bits).reshape(shp), bits.reshape(shp)
    return a, None


@dataclasses.dataclass
class Weights:
    shape: ModelShape
    seed: int
    values: dict  # name -> float32 array (bf16-exact for bf16 models)
    bits: dict    # name -> uint16 bf16 bit patterns (bf16 models only)

    def __getitem__(self, name):
        return self.values[name]


def make_weights(shape: ModelShape, seed: int = 0, threads: int = 8) -> Weights:
    """Every tensor i of the canonical order is drawn from its own stream
    PCG64(SeedSequence([seed, i])), so tensors can be drawn in parallel."""
    specs = tensor_specs(shape)
    with ThreadPoolExecutor(max(1, threads)) as ex:
        out = list(ex.map(lambda it: _draw(seed, it[0], it[1][1], it[1][2], shape.dtype),
                          enumerate(specs)))
    values, bits = {}, {}
    for (name, _, _), (v, b) in zip(specs, out):
        values[name] = v
        if b is not None:
            bits[name] = b
    return Weights(shape, seed, values, bits)


# ----------------------------------------------------------------------------
# weight blob (the byte format whisper_ctx_create reads; see the C header)
# ----------------------------------------------------------------------------

BLOB_MAGIC = b"WHSPMI01"
BLOB_HEADER_BYTES = 256
BLOB_ALIGN = 256


def blob_layout(shape: ModelShape):
    """(name, shape, byte offset) per tensor, plus the total size."""
    esz = 4 if shape.dtype == "f32" else 2
    off = BLOB_HEADER_BYTES
    lay = []
    for name, shp, _ in tensor_specs(shape):
        lay.append((name, shp, off))
        off += int(np.prod(shp)) * esz
        off = (off + BLOB_ALIGN - 1) // BLOB_ALIGN * BLOB_ALIGN
    return lay, off


def pack_blob(w: Weights) -> np.ndarray:
    s = w.shape
    lay, total = blob_layout(s)
    buf = np.zeros(total, dtype=np.uint8)
    hdr = struct.pack(
        "<8s14i", BLOB_MAGIC, 1, 0 if s.dtype == "f32" else 1,
        s.n_mels, s.n_audio_ctx, s.d, s.n_head, s.n_enc,
        s.n_vocab, s.n_text_ctx, s.d, s.n_head, s.n_dec, len(lay), 0)
    buf[:len(hdr)] = np.frombuffer(hdr, dtype=np.uint8)
    for name, shp, off in lay:
        src = w.bits[name] if s.dtype == "bf16" else w.values[name]
        raw = np.ascontiguousarray(src).view(np.uint8).reshape(-1)
        buf[off:off + raw.size] = raw
    return buf


# ----------------------------------------------------------------------------
# audio segments and workloads
# ----------------------------------------------------------------------------

@dataclasses.dataclass
class Segment:
    audio: np.ndarray        # float32, 16 kHz mono, 1..480000 samples
    user_id: int
    segment_id: int
    prompt: list
    max_new_tokens: int
    arrival_us: int = 0

    @property
    def seconds(self) -> float:
        return self.audio.size / SAMPLE_RATE


def synth_audio(rng: np.random.Generator, n_samples: int) -> np.ndarray:
    """Three sinusoids, f ~ U(100, 4000) Hz, amplitude ~ U(0.1, 0.3),
    phase ~ U(0, 2 pi), plus N(0, 0.05^2) noise."""
    f = rng.uniform(100.0, 4000.0, 3)
    a = rng.uniform(0.1, 0.3, 3)
    ph = rng.uniform(0.0, 2 * np.pi, 3)
    t = np.arange(n_samples, dtype=np.float64) / SAMPLE_RATE
    x = np.zeros(n_samples, dtype=np.float64)
    for i in range(3):
        x += a[i] * np.sin(2 * np.pi * f[i] * t + ph[i])
    x += rng.normal(0.0, 0.05, n_samples)
    return x.astype(np.float32)


def length_samples(rng: np.random.Generator, lo_s=3.0, hi_s=30.0) -> int:
    return int(round(rng.uniform(lo_s, hi_s) * SAMPLE_RATE))


def fixed_batch(shape: ModelShape, lengths, n_new, seed: int = 1) -> list:
    rng = np.random.Generator(np.random.PCG64(seed))
    p = prompt_for(shape)
    segs = []
    for i, n in enumerate(lengths):
        nn = n_new[i] if isinstance(n_new, (list, tuple, np.ndarray)) else n_new
        segs.append(Segment(synth_audio(rng, int(n)), 0, i, list(p), int(nn), 0))
    return segs


def uniform_batch(shape: ModelShape, n_seg: int, n_new, seed: int = 1) -> list:
    rng = np.random.Generator(np.random.PCG64(seed))
    lengths = [length_samples(rng) for _ in range(n_seg)]
    return fixed_batch(shape, lengths, n_new, seed=seed + 1000)


def poisson_users(shape: ModelShape, n_users: int, n_seg: int, mean_gap_s: float,
                  new_lo: int, new_hi: int, seed: int = 1) -> list:
    """n_users users, each with exponential inter-arrival gaps (mean
    mean_gap_s); the first n_seg arrivals over all users form the workload.
    Output lengths are uniform integers on [new_lo, new_hi]."""
    rng = np.random.Generator(np.random.PCG64(seed))
    per_user = n_seg // n_users + 8
    events = []
    for u in range(n_users):
        t = np.cumsum(rng.exponential(mean_gap_s, per_user))
        for k in range(per_user):
            events.append((float(t[k]), u, k))
    events.sort()
    events = events[:n_seg]
    p = prompt_for(shape)
    segs = []
    for (t, u, k) in events:
        n = length_samples(rng)
        segs.append(Segment(synth_audio(rng, n), u, u * 1_000_000 + k, list(p),
                            int(rng.integers(new_lo, new_hi + 1)), int(round(t * 1e6))))
    return segs


# The five workloads: (model shape, segment list factory, decode slots).
def workload(name: str, seed: int = 1):
    if name == "tiny-b2":
        s = TINY
        return s, fixed_batch(s, [48000, 112000], 16, seed), 2
    if name == "base-b16":
        s = BASE
        return s, uniform_batch(s, 16, 64, seed), 16
    if name == "small-u8-b64":
        s = SMALL
        return s, poisson_users(s, 8, 64, 5.0, 16, 128, seed), 64
    if name == "large-v3-b32":
        s = LARGE_V3
        return s, uniform_batch(s, 32, 224, seed), 32
    if name == "turbo-u64-q512":
        s = TURBO
        return s, poisson_users(s, 64, 512, 5.0, 16, 224, seed), 128
    if name == "ctc-tiny-b2":
        s = CTC_TINY
        return s, fixed_batch(s, [48000, 112000], 1500, seed), 2
    if name == "ctc-base-u64-q512":
        # the turbo queue's arrivals and lengths, served by an encoder-only
        # CTC model (output capacity 1500 labels, one per encoder frame)
        s = CTC_BASE
        segs = poisson_users(s, 64, 512, 5.0, 16, 224, seed)
        for g in segs:
            g.max_new_tokens = 1500
        return s, segs, 32
    raise KeyError(name)


WORKLOADS = ("tiny-b2", "base-b16", "small-u8-b64", "large-v3-b32", "turbo-u64-q512", "ctc-tiny-b2",
             "ctc-base-u64-q512")


def recording(shape: ModelShape, rng: np.random.Generator, seconds: float, user_id: int, first_id: int,
              arrival_us: int = 0, tokens_per_s: float = 3.3) -> list:
    """One user's recording of `seconds` cut into VAD-style segments of 3-30 s
    (lengths drawn uniformly, the last one taking the remainder), each with
    the standard prompt and max(4, round(tokens_per_s * length)) tokens (at
    most 224): dictation speed of about 2.5 words per second. Every segment
    arrives with the recording."""
    p = prompt_for(shape)
    left = float(seconds)
    lengths = []
    while left > 30.0:
        L = float(rng.uniform(3.0, min(30.0, left - 3.0)))
        lengths.append(L)
        left -= L
    lengths.append(left)
    segs = []
    for k, L in enumerate(lengths):
        n = int(round(L * SAMPLE_RATE))
        nt = int(min(224, max(4, round(tokens_per_s * L))))
        segs.append(Segment(synth_audio(rng, n), user_id, first_id + k, list(p), nt, int(arrival_us)))
    return segs
