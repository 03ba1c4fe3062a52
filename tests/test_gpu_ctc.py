"""GPU parity of the encoder-only CTC variant (greedy best-path decoding
and prefix beam search) against the float64 oracle (oracle/ctc.py), through
the C ABI.

Tolerances: head logits per frame relative to the frame's largest
magnitude, 1e-3 for the fp32 model and 2e-2 for bf16 (the decoder logits'
bar). The device's per-frame ids equal the argmax of its own logits
exactly; they equal the oracle's on every frame whose top-1 - top-2 margin
exceeds twice the frame's measured logit error, and otherwise lie within
that band (tests/parity.py). The device's labels equal the oracle's CTC
collapse of the device's ids, always; so they equal the oracle's labels
whenever no frame is a near tie."""
import copy
import sys

import numpy as np
import pytest

import oracle
from oracle import ctc as OC
from oracle import model as M
from paper_2507_01021_amd import binding, synth

from parity import TOL, check_ctc_entry

pytestmark = pytest.mark.gpu


def log(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def _oracle(W, shape, segs, pad_mode=0):
    return OC.transcribe_ctc(W, shape, segs, pad_mode=pad_mode, return_logits=True)


def _check_labels(seg, ref, ids, near, labels):
    """Labels: the oracle's collapse of the device's ids; with no near-tie
    frame, the oracle's own labels."""
    assert labels == OC.collapse(ids.tolist())[:seg.max_new_tokens]
    if near == 0:
        assert labels == ref["tokens"]


@pytest.fixture(scope="module")
def tiny():
    shape, segs, slots = synth.workload("ctc-tiny-b2")
    W = synth.make_weights(shape, 0)
    ref = _oracle(W, shape, segs)
    with binding.Context(synth.pack_blob(W), max_slots=2) as ctx:
        yield shape, W, segs, ref, ctx


def test_ctc_tiny_logits_ids_labels(tiny):
    shape, W, segs, ref, ctx = tiny
    log("ctc-tiny: encode 2 segments")
    ctx.encode(segs, [0, 1])
    got = []
    for b, (s, r) in enumerate(zip(segs, ref)):
        mel = ctx.debug_copy(binding.T_MEL, b, (shape.n_mels, 3000))
        assert np.abs(mel - oracle.log_mel_segment(s.audio, shape.n_mels)).max() < 2e-5
        got.append(check_ctc_entry(ctx, shape, b, s, r, TOL["f32"], log))
    res = ctx.transcribe(segs)
    for s, r, g, (ids, near) in zip(segs, ref, res, got):
        log(f"segment {s.segment_id}: {len(r['tokens'])} labels (oracle), {g['tokens'].size} (device)")
        assert g["status"] == 0 and g["tokens"].size <= s.max_new_tokens
        _check_labels(s, r, ids, near, g["tokens"].tolist())
    assert any(near == 0 for _, near in got)     # the exact-label case occurs


def test_ctc_base_bf16_and_queue():
    """bf16 model: per-entry parity on a pass of 3 segments (logits, ids, and
    labels as the collapse of the ids), then a queue of 40 segments in passes
    of 16: every result maps back to its segment and equals the segment's
    labels from the solo pass (bit-exact); a small max_new_tokens truncates."""
    shape = synth.CTC_BASE
    W = synth.make_weights(shape, 0)
    segs = synth.uniform_batch(shape, 3, 1500, seed=3)
    ref = _oracle(W, shape, segs)
    with binding.Context(synth.pack_blob(W), max_slots=16, max_encode_batch=16) as ctx:
        log("ctc-base: encode 3 segments")
        ctx.encode(segs, list(range(3)))
        got = [check_ctc_entry(ctx, shape, b, s, r, TOL["bf16"], log) for b, (s, r) in enumerate(zip(segs, ref))]
        solo = [ctx.transcribe([s])[0]["tokens"] for s in segs]
        for s, t, r, (ids, near) in zip(segs, solo, ref, got):
            _check_labels(s, r, ids, near, t.tolist())
        q = []
        for k in range(40):
            t = copy.copy(segs[k % 3])
            t.segment_id = 1000 + k
            t.user_id = k % 5
            t.arrival_us = (k * 7919) % 41
            t.max_new_tokens = 1500 if k % 7 else 3
            q.append(t)
        log("ctc-base: queue of 40 segments, passes of 16")
        res = ctx.transcribe(q)
        for k, (t, r) in enumerate(zip(q, res)):
            assert (r["segment_id"], r["user_id"], r["status"]) == (t.segment_id, t.user_id, 0)
            want = solo[k % 3][: t.max_new_tokens]
            assert np.array_equal(r["tokens"], want)
        served = ctx.transcribe(q, realtime=True)
        for a, b in zip(res, served):
            assert np.array_equal(a["tokens"], b["tokens"])


def test_ctc_frames_without_a_finite_logit_raise():
    """A head whose logits are all NaN (or all -inf) has no best-path id
    for any frame: the device records the blank for such frames and the
    call that reads the batch fails with a device error naming the cause,
    instead of returning an id outside the vocabulary."""
    shape, segs, slots = synth.workload("ctc-tiny-b2")
    for bad in (np.nan, -np.inf):
        W = synth.make_weights(shape, 0)
        W.values["ctc.b"] = np.full_like(W.values["ctc.b"], bad)
        with binding.Context(synth.pack_blob(W), max_slots=2) as ctx:
            with pytest.raises(binding.WhisperError) as e:
                ctx.transcribe(segs)
        log(f"head bias {bad}: {e.value}")
        assert e.value.status == binding.E_DEVICE and "finite logit" in str(e.value)


def test_ctc_decoder_calls_refused(tiny):
    shape, W, segs, ref, ctx = tiny
    with pytest.raises(binding.WhisperError):
        ctx.decode_step([0], logits=True)
    with pytest.raises(binding.WhisperError):
        ctx.time_kernel(binding.K_CROSS_ATTN, 1, 1)


@pytest.mark.parametrize("beam,scale", [(2, 30.0), (4, 30.0), (8, 30.0), (4, 1.0)])
def test_ctc_prefix_beam_search_matches_oracle(beam, scale):
    """ctc_beam >= 2: the GPU's prefix beam search against the oracle's on
    the fp32 tiny model, with the head's weights scaled by `scale`. With a
    peaked head (scale 30) the pruning decisions are clear-cut and the labels
    must be identical wherever the oracle's smallest pruning margin exceeds
    1e-2 nats. With the plain head many decisions are near ties; the labels
    must then be identical or the margin must lie within 5e-3 nats, the
    budget of fp32 scores summed over up to 350 frames."""
    shape, segs, slots = synth.workload("ctc-tiny-b2")
    W = synth.make_weights(shape, 0)
    W.values["ctc.w"] = (W.values["ctc.w"] * np.float32(scale)).astype(np.float32)
    ref = OC.transcribe_ctc(W, shape, segs, beam=beam)
    with binding.Context(synth.pack_blob(W), max_slots=2, ctc_beam=beam) as ctx:
        res = ctx.transcribe(segs)
        solo = [ctx.transcribe([s])[0] for s in segs]
    same = 0
    for s, r, g, g1 in zip(segs, ref, res, solo):
        eq = g["tokens"].tolist() == r["tokens"]
        log(f"beam {beam}, scale {scale}, segment {s.segment_id}: {len(r['tokens'])} labels (oracle), "
            f"{g['tokens'].size} (device), margin {r['margin']:.3g}, identical {eq}")
        assert np.array_equal(g["tokens"], g1["tokens"])          # batch = solo
        assert g["status"] == 0 and all(1 <= c < shape.n_vocab for c in g["tokens"])
        if scale > 1 and r["margin"] > 1e-2:
            assert eq
        if not eq:
            assert r["margin"] < 5e-3
        same += eq
    if scale > 1:
        assert same == len(segs)


def test_ctc_beam_base_bf16_matches_oracle_under_margin_rule():
    """bf16 prefix beam search (beam 4) against the oracle's search on its
    float64 logits. A segment's device labels must equal the oracle's unless
    the oracle's smallest pruning margin is within the error budget of the
    device's scores: a prefix's score is a sum over frames of log-softmax
    terms, each off by at most twice the frame's largest logit error, so two
    prefixes' difference moves by at most 4 times the sum of those errors
    (plus 5e-3 nats for fp32 summation). Also batch = solo, valid ids."""
    shape = synth.CTC_BASE
    W = synth.make_weights(shape, 0)
    W.values["ctc.w"] = (W.values["ctc.w"] * np.float32(30.0)).astype(np.float32)
    W.bits["ctc.w"] = synth.round_to_bf16(W.values["ctc.w"])
    W.values["ctc.w"] = synth.bf16_to_f32(W.bits["ctc.w"]).reshape(W.values["ctc.w"].shape)
    segs = synth.fixed_batch(shape, [16000, 24000, 48000, 64000], 1500, seed=5)
    ref = OC.transcribe_ctc(W, shape, segs, beam=4, return_logits=True)
    blob = synth.pack_blob(W)
    with binding.Context(blob, max_slots=4) as greedy_ctx:       # the device's logits of each entry
        greedy_ctx.encode(segs, list(range(4)))
        lgs = [greedy_ctx.debug_copy(binding.T_CTC_LOGITS, b, (1500, shape.n_vocab)) for b in range(4)]
    with binding.Context(blob, max_slots=4, ctc_beam=4) as ctx:
        res = ctx.transcribe(segs)
        solo = [ctx.transcribe([s])[0] for s in segs]
    checked = 0
    for s, r, g, g1, lg in zip(segs, ref, res, solo, lgs):
        T = OC.valid_frames(s.audio.size)
        err = np.abs(lg[:T] - r["logits"][:T]).max(axis=1)
        assert (err / np.abs(r["logits"][:T]).max(axis=1)).max() < TOL["bf16"]
        budget = 4.0 * float(err.sum()) + 5e-3
        eq = g["tokens"].tolist() == r["tokens"]
        log(f"bf16 beam 4, segment {s.segment_id}: {T} frames, {len(r['tokens'])} labels (oracle), "
            f"{g['tokens'].size} (device), margin {r['margin']:.3g}, budget {budget:.3g}, identical {eq}")
        assert np.array_equal(g["tokens"], g1["tokens"])          # batch = solo
        assert g["status"] == 0 and all(1 <= c < shape.n_vocab for c in g["tokens"])
        if r["margin"] > budget:
            assert eq
            checked += 1
    log(f"bf16 beam: {checked} of {len(segs)} segments beyond the error budget")


def test_ctc_beam_base_bf16_runs_and_is_batch_independent():
    shape = synth.CTC_BASE
    W = synth.make_weights(shape, 0)
    segs = synth.uniform_batch(shape, 4, 1500, seed=5)
    with binding.Context(synth.pack_blob(W), max_slots=4, ctc_beam=4) as ctx:
        res = ctx.transcribe(segs)
        solo = [ctx.transcribe([s])[0] for s in segs]
    for s, g, g1 in zip(segs, res, solo):
        assert np.array_equal(g["tokens"], g1["tokens"])
        assert 0 < g["tokens"].size <= OC.valid_frames(s.audio.size)
        assert all(1 <= c < shape.n_vocab for c in g["tokens"])
