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

Beam search is a decoding variant of the same model: CTC prefix beam search
(no language model), after Hannun et al.'s prefix search, with the
per-frame candidates pruned to the most likely labels.
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


def transcribe_ctc(W, shape, segments, pad_mode=0, return_logits=False, beam=0):
    """One batched call: features of every segment on the 30 s window,
    stacked, one encoder pass, the CTC head, then greedy decoding of each
    segment over its own frames (beam >= 2: prefix beam search with that
    beam and as many candidate ids per frame). A segment keeps at most
    max_new_tokens labels (its output capacity).

    Returns one dict per input segment, in input order:
    {user_id, segment_id, tokens, ids[, margin][, logits]}."""
    if len(segments) == 0:
        return []
    feats = np.stack([log_mel_segment(s.audio, shape.n_mels, pad_mode) for s in segments])
    L = ctc_logits(W, encoder(W, shape, feats))
    out = []
    for b, s in enumerate(segments):
        T = valid_frames(len(s.audio))
        ids = best_path(L[b], T)
        r = {"user_id": s.user_id, "segment_id": s.segment_id, "ids": ids,
             "tokens": collapse(ids)[:s.max_new_tokens]}
        if beam >= 2:
            labels, r["margin"] = prefix_beam_search(L[b], T, beam, beam)
            r["tokens"] = labels[:s.max_new_tokens]
        if return_logits:
            r["logits"] = L[b]
        out.append(r)
    return out


# ----------------------------------------------------------------------------
# prefix beam search (a decoding variant of the same model)
# ----------------------------------------------------------------------------

def _lae(a, b):
    """log(exp a + exp b) with -inf handled."""
    if a == -math.inf:
        return b
    if b == -math.inf:
        return a
    m = max(a, b)
    return m + math.log(math.exp(a - m) + math.exp(b - m))


def frame_candidates(logits_t, per_frame):
    """Log-probabilities of one frame (log-softmax over the vocabulary), the
    blank's, and the per_frame most likely non-blank ids (lowest id on
    ties) with theirs."""
    lg = np.asarray(logits_t, dtype=np.float64)
    m = lg.max()
    lp = lg - (m + math.log(np.exp(lg - m).sum()))
    order = sorted(range(1, lg.size), key=lambda c: (-lp[c], c))[:per_frame]
    return float(lp[BLANK]), [(c, float(lp[c])) for c in order]


def prefix_beam_search(logits, n_frames, beam, per_frame):
    """CTC prefix beam search without a language model over frames
    0..n_frames-1. Every kept prefix carries the log-probability of the
    paths that end in a blank (pb) and of those that end in its last label
    (pnb). At each frame a prefix
      * stays the same through the blank (to pb, from pb + pnb),
      * stays the same through its own last label, from pnb (a repeat),
      * grows by a label c among the frame's per_frame candidates: from
        pb + pnb, or from pb only when c is its last label (a blank must
        separate a repeated label);
    equal prefixes are merged by adding probabilities. The `beam` most
    probable prefixes (pb + pnb) survive; ties go to the earlier candidate
    in the order: every kept prefix's "stay" in beam order, then its
    extensions, beam by beam, in candidate order. The most probable final
    prefix is the output.

    Returns (labels, margin): margin is the smallest gap, in log-probability,
    between the last surviving and the first dropped candidate over all
    frames, and between the best and second-best final prefixes (inf when
    nothing was ever dropped and a single prefix remains)."""
    beams = [((), 0.0, -math.inf)]             # (prefix, pb, pnb), in beam order
    margin = math.inf
    for t in range(n_frames):
        lpb, cands = frame_candidates(logits[t], per_frame)
        nxt = {}                               # prefix -> [pb, pnb, candidate rank]
        rank = 0

        def add(prefix, pb, pnb):
            nonlocal rank
            if prefix not in nxt:
                nxt[prefix] = [-math.inf, -math.inf, rank]
                rank += 1
            e = nxt[prefix]
            e[0] = _lae(e[0], pb)
            e[1] = _lae(e[1], pnb)

        for prefix, pb, pnb in beams:          # stays first, in beam order
            tot = _lae(pb, pnb)
            stay_nb = pnb + dict(cands).get(prefix[-1], -math.inf) if prefix else -math.inf
            add(prefix, tot + lpb, stay_nb)
        for prefix, pb, pnb in beams:          # then extensions
            tot = _lae(pb, pnb)
            for c, lpc in cands:
                src = pb if (prefix and c == prefix[-1]) else tot
                add(prefix + (c,), -math.inf, src + lpc)
        ranked = sorted(nxt.items(), key=lambda kv: (-_lae(kv[1][0], kv[1][1]), kv[1][2]))
        if len(ranked) > beam:
            margin = min(margin, _lae(*ranked[beam - 1][1][:2]) - _lae(*ranked[beam][1][:2]))
        beams = [(p, e[0], e[1]) for p, e in ranked[:beam]]
    if len(beams) > 1:
        margin = min(margin, _lae(beams[0][1], beams[0][2]) - _lae(beams[1][1], beams[1][2]))
    return list(beams[0][0]), margin
