"""GPU edge cases against the oracle, through the C ABI: the empty call, the
shortest and longest segments (1 and 480000 samples), a decode that fills
the text context to its last position (4 prompt tokens + 444 new = 448, in
the fp32 and the bf16 model), the model widths (bf16 and fp32), mel channel
counts and small vocabularies no workload uses, for the
encoder-decoder and the CTC variant (1 and 1500 frames). Tolerances as in
test_gpu_parity."""
import sys

import numpy as np
import pytest

import oracle
from oracle import ctc as OC
from paper_2507_01021_amd import binding, synth

from parity import (TOL, check_ctc_entry, check_tokens, drive_teacher_forced, float64_weights, oracle_run,
                    rel_row_err)

pytestmark = pytest.mark.gpu


def log(*a):
    print(*a, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def tiny():
    shape = synth.TINY
    W = synth.make_weights(shape, 0)
    with binding.Context(synth.pack_blob(W), max_slots=4) as ctx:
        yield shape, W, ctx


def test_empty_call(tiny):
    shape, W, ctx = tiny
    assert ctx.transcribe([]) == []
    assert ctx.transcribe([], realtime=True) == []


def test_shortest_and_longest_segments(tiny):
    shape, W, ctx = tiny
    segs = synth.fixed_batch(shape, [1, 480000], 8, seed=11)
    ref = oracle_run(W, shape, segs, n_new=8)
    log("tiny: encode segments of 1 and 480000 samples")
    ctx.encode(segs, [0, 1])
    for i, r in enumerate(ref):
        mel = ctx.debug_copy(binding.T_MEL, i, (shape.n_mels, 3000))
        assert np.abs(mel - r["mel"]).max() < 2e-5
        E = ctx.debug_copy(binding.T_ENC_OUT, i, (1500, shape.d))
        assert rel_row_err(E, r["E"]).max() < TOL["f32"]
    toks, lgs = drive_teacher_forced(ctx, [0, 1], segs, ref, 8)
    for k in range(2):
        assert rel_row_err(lgs[k], ref[k]["logits"]).max() < TOL["f32"]
        check_tokens(toks[k], ref[k]["logits"], gpu_logits=lgs[k], min_strict=4)


def test_decode_to_the_last_text_position(tiny):
    """n_prompt + max_new_tokens = 448: the self-attention caches fill up."""
    shape, W, ctx = tiny
    n_new = shape.n_text_ctx - 4
    segs = synth.fixed_batch(shape, [32000, 96000], n_new, seed=12)
    ref = oracle_run(W, shape, segs, n_new=n_new)
    log(f"tiny: teacher-forced decode of {n_new} tokens in 2 slots")
    ctx.encode(segs, [2, 3])
    toks, lgs = drive_teacher_forced(ctx, [2, 3], segs, ref, n_new)
    for k in range(2):
        e = rel_row_err(lgs[k], ref[k]["logits"])
        log(f"slot {k}: logits rel err max {e.max():.2e} (last position {e[-1]:.2e})")
        assert e.max() < TOL["f32"]
        check_tokens(toks[k], ref[k]["logits"], gpu_logits=lgs[k], min_strict=n_new // 2)
    with pytest.raises(binding.WhisperError):  # the slots retired with their last token
        ctx.decode_step([2])
    res = ctx.transcribe(segs)
    for r, s in zip(res, segs):
        assert r["tokens"].size == n_new


def test_bf16_decode_to_the_last_text_position():
    """The bf16 decode path (base shape) filled to position 447: the
    self-attention kernel's P·V over more than 256 cached positions (a
    second batch of V rows per wave), the cache appends and the head at every
    position, against the oracle under teacher forcing."""
    shape = synth.BASE
    W = synth.make_weights(shape, 0)
    n_new = shape.n_text_ctx - 4
    segs = synth.fixed_batch(shape, [64000, 288000], n_new, seed=13)
    log(f"base: oracle decode of {n_new} tokens for 2 segments")
    ref = oracle_run(float64_weights(W), shape, segs, n_new=n_new)
    with binding.Context(synth.pack_blob(W), max_slots=2) as ctx:
        log(f"base: teacher-forced decode of {n_new} tokens in 2 slots")
        ctx.encode(segs, [0, 1])
        toks, lgs = drive_teacher_forced(ctx, [0, 1], segs, ref, n_new)
        for k in range(2):
            e = rel_row_err(lgs[k], ref[k]["logits"])
            strict, near = check_tokens(toks[k], ref[k]["logits"], gpu_logits=lgs[k], min_strict=n_new // 2)
            log(f"slot {k}: logits rel err max {e.max():.2e} (last position {e[-1]:.2e}), "
                f"tokens strict {strict} near-tie {near}")
            assert e.max() < TOL["bf16"]


@pytest.mark.parametrize("d", [1024, 1536, 2048])
def test_widths_without_a_workload(d):
    """Model widths the library accepts that no workload uses (1024 is
    Whisper medium's, 2048 the largest allowed; with the workloads' 384,
    512, 768 and 1280 every supported width runs), bf16, one encoder and two
    decoder layers with the full vocabulary: encoder output, teacher-forced
    logits and tokens of one segment against the oracle."""
    shape = synth.BASE.with_(name=f"w{d}", d=d, n_head=d // 64, n_enc=1, n_dec=2)
    W = synth.make_weights(shape, 0)
    segs = synth.fixed_batch(shape, [400000], 8, seed=14)
    log(f"width {d}: oracle")
    ref = oracle_run(float64_weights(W), shape, segs, n_new=8)
    with binding.Context(synth.pack_blob(W), max_slots=1) as ctx:
        log(f"width {d}: encode and teacher-forced decode")
        ctx.encode(segs, [0])
        E = ctx.debug_copy(binding.T_ENC_OUT, 0, (1500, d))
        ee = rel_row_err(E, ref[0]["E"]).max()
        toks, lgs = drive_teacher_forced(ctx, [0], segs, ref, 8)
        e = rel_row_err(lgs[0], ref[0]["logits"])
        strict, near = check_tokens(toks[0], ref[0]["logits"], gpu_logits=lgs[0], min_strict=4)
        log(f"width {d}: encoder rel err {ee:.2e}, logits rel err max {e.max():.2e}, "
            f"tokens strict {strict} near-tie {near}")
        assert ee < TOL["bf16"] and e.max() < TOL["bf16"]


@pytest.mark.parametrize("d", [512, 1280, 2048])
def test_fp32_model_widths(d):
    """The fp32 model (SIMT GEMMs, fp32 caches) beyond the tiny width:
    encoder output and teacher-forced logits and tokens of one segment
    against the oracle at the fp32 tolerance (one encoder and two decoder
    layers, full vocabulary)."""
    shape = synth.TINY.with_(name=f"f{d}", d=d, n_head=d // 64, n_enc=1, n_dec=2)
    W = synth.make_weights(shape, 0)
    segs = synth.fixed_batch(shape, [240000], 8, seed=17)
    ref = oracle_run(float64_weights(W), shape, segs, n_new=8)
    with binding.Context(synth.pack_blob(W), max_slots=1) as ctx:
        log(f"fp32 width {d}: encode and teacher-forced decode")
        ctx.encode(segs, [0])
        E = ctx.debug_copy(binding.T_ENC_OUT, 0, (1500, d))
        ee = rel_row_err(E, ref[0]["E"]).max()
        toks, lgs = drive_teacher_forced(ctx, [0], segs, ref, 8)
        e = rel_row_err(lgs[0], ref[0]["logits"]).max()
        check_tokens(toks[0], ref[0]["logits"], gpu_logits=lgs[0], min_strict=6)
        log(f"fp32 width {d}: encoder rel err {ee:.2e}, logits rel err {e:.2e}")
        assert ee < TOL["f32"] and e < TOL["f32"]


@pytest.mark.parametrize("n_mels", [4, 68, 100])
def test_mel_counts_without_a_workload(n_mels):
    """Mel channel counts the library accepts besides Whisper's 80 and 128
    (multiples of 4 up to 128): log-mel features, encoder output and
    teacher-forced logits of one segment against the oracle (bf16, base
    width, one encoder and one decoder layer)."""
    shape = synth.BASE.with_(name=f"m{n_mels}", n_mels=n_mels, n_enc=1, n_dec=1)
    W = synth.make_weights(shape, 0)
    segs = synth.fixed_batch(shape, [200000], 6, seed=15)
    ref = oracle_run(float64_weights(W), shape, segs, n_new=6)
    with binding.Context(synth.pack_blob(W), max_slots=1) as ctx:
        log(f"{n_mels} mel channels: encode and teacher-forced decode")
        ctx.encode(segs, [0])
        mel = ctx.debug_copy(binding.T_MEL, 0, (n_mels, 3000))
        me = np.abs(mel - ref[0]["mel"]).max()
        E = ctx.debug_copy(binding.T_ENC_OUT, 0, (1500, shape.d))
        ee = rel_row_err(E, ref[0]["E"]).max()
        toks, lgs = drive_teacher_forced(ctx, [0], segs, ref, 6)
        e = rel_row_err(lgs[0], ref[0]["logits"]).max()
        check_tokens(toks[0], ref[0]["logits"], gpu_logits=lgs[0], min_strict=3)
        log(f"{n_mels} mel channels: mel abs err {me:.1e}, encoder rel err {ee:.2e}, logits rel err {e:.2e}")
        assert me < 2e-5 and ee < TOL["bf16"] and e < TOL["bf16"]


@pytest.mark.parametrize("n_vocab", [1, 33, 1000])
def test_small_vocabularies(n_vocab):
    """Decoder vocabularies far below Whisper's, down to a single id (the
    last 32-id tile of the head ragged or alone): teacher-forced logits and
    greedy tokens of two segments against the oracle (bf16, base width, one
    encoder and two decoder layers, prompts of in-range ids)."""
    shape = synth.BASE.with_(name=f"v{n_vocab}", n_vocab=n_vocab, n_enc=1, n_dec=2)
    W = synth.make_weights(shape, 0)
    segs = synth.fixed_batch(shape, [48000, 160000], 8, seed=16)
    for k, sg in enumerate(segs):
        sg.prompt = [(3 * k + j) % n_vocab for j in range(3)]
    ref = oracle_run(float64_weights(W), shape, segs, n_new=8)
    with binding.Context(synth.pack_blob(W), max_slots=2) as ctx:
        log(f"vocabulary {n_vocab}: encode and teacher-forced decode")
        ctx.encode(segs, [0, 1])
        toks, lgs = drive_teacher_forced(ctx, [0, 1], segs, ref, 8)
        for k in range(2):
            e = rel_row_err(lgs[k], ref[k]["logits"]).max()
            log(f"vocabulary {n_vocab} slot {k}: logits rel err {e:.2e}")
            assert e < TOL["bf16"]
            assert np.all((np.asarray(toks[k]) >= 0) & (np.asarray(toks[k]) < n_vocab))
            if n_vocab > 1:
                check_tokens(toks[k], ref[k]["logits"], gpu_logits=lgs[k], min_strict=4)
        res = ctx.transcribe(segs)
        for r, sg in zip(res, segs):
            assert r["tokens"].size == sg.max_new_tokens
            assert np.all((r["tokens"] >= 0) & (r["tokens"] < n_vocab))


def test_ctc_shortest_and_longest_segments():
    """CTC segments of 1 sample (one frame) and 30 s (all 1500 frames):
    logits, per-frame ids and labels against the oracle."""
    shape = synth.CTC_TINY
    W = synth.make_weights(shape, 0)
    segs = synth.fixed_batch(shape, [1, 480000], 1500, seed=13)
    ref = OC.transcribe_ctc(W, shape, segs, return_logits=True)
    with binding.Context(synth.pack_blob(W), max_slots=2) as ctx:
        ctx.encode(segs, [0, 1])
        ids = []
        for b, (s, r) in enumerate(zip(segs, ref)):
            T = OC.valid_frames(s.audio.size)
            assert T == (1 if s.audio.size == 1 else 1500)
            ids.append(check_ctc_entry(ctx, shape, b, s, r, TOL["f32"], log)[0])
        res = ctx.transcribe(segs)
        for s, r, g, i in zip(segs, ref, res, ids):
            log(f"ctc-tiny: {s.audio.size} samples, {i.size} frames, {g['tokens'].size} labels")
            assert g["status"] == 0
            assert g["tokens"].tolist() == OC.collapse(i.tolist())[:s.max_new_tokens]
