"""CTC head and greedy (best-path) decoding, in float64.

TEST INFRASTRUCTURE ONLY (see oracle/__init__.py).

The paper notes that the same multiplexing serves encoder-only recognisers
decoded with connectionist temporal classification, since they have no
dependency between segments either (Introduction; the closing remark of
Section 2.3). It names no such model. The model read here is the Whisper
encoder of oracle.model followed by a linear head to a vocabulary whose id 0
is the CTC blank. Greedy decoding, Graves et al.'s best-path decoding:
* take the most likely id of every encoder frame that covers the segment's
  audio (lowest id on ties);
* merge runs of the same id;
* drop blanks.
An encoder frame covers 320 samples: a 160-sample hop, then the stride-2
convolution.
"""
import math

import numpy as np

from .frontend import log_mel_segment
from .model import encoder

BLANK = 0
SAMPLES_PER_FRAME = 320
N_FRAMES = 1500


def valid_frames(n_samples):
    """Encoder frames that cover n_samples of audio: ceil(n / 320), at most 1500."""
    return min(N_FRAMES, int(math.ceil(n_samples / SAMPLES_PER_FRAME)))


def ctc_logits(W, E):
    """Per-frame vocabulary scores: E W_ctc^T + b_ctc (E [..., frames, d])."""
    w = np.asarray(W["ctc.w"], dtype=np.float64)
    b = np.asarray(W["ctc.b"], dtype=np.float64)
    return np.asarray(E, dtype=np.float64) @ w.T + b


def best_path(logits, n_frames):
    """The most likely id of each of the first n_frames frames (first maximum,
    i.e. the lowest id, on ties)."""
    return [int(np.argmax(logits[t])) for t in range(n_frames)]


def collapse(ids, blank=BLANK):
    """The CTC map from a frame path to a label sequence: merge each run of
    equal ids into one, then remove blanks."""
    out = []
    prev = None
    for i in ids:
        if i != prev and i != blank:
            out.append(int(i))
        prev = i
    return out


def transcribe_ctc(W, shape, segments, pad_mode=0, return_logits=False):
    """One batched call: features of every segment on the 30 s window,
    stacked, one encoder pass, the CTC head, then greedy decoding of each
    segment over its own frames. A segment keeps at most max_new_tokens
    labels (its output capacity).

    Returns one dict per input segment, in input order:
    {user_id, segment_id, tokens, ids[, logits]}."""
    if len(segments) == 0:
        return []
    feats = np.stack([log_mel_segment(s.audio, shape.n_mels, pad_mode) for s in segments])
    L = ctc_logits(W, encoder(W, shape, feats))
    out = []
    for b, s in enumerate(segments):
        ids = best_path(L[b], valid_frames(len(s.audio)))
        r = {"user_id": s.user_id, "segment_id": s.segment_id, "ids": ids,
             "tokens": collapse(ids)[:s.max_new_tokens]}
        if return_logits:
            r["logits"] = L[b]
        out.append(r)
    return out
