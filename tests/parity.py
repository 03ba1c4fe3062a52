"""Shared parity helpers for the GPU tests: the tolerance rules for logits
and greedy tokens, and oracle runs on the same seeded inputs.

Greedy tokens (the greedy choice of Listing 1's generate, lowest id on
ties). At every teacher-forced position the GPU returns its argmax together
with the logits it took the argmax of. Write err = max_j |g_j - o_j| for
that row (g the GPU's logits, o the oracle's). When the oracle's top-1
beats its top-2 by more than band = 2 err, no id can overtake the top-1 on
the GPU, so the GPU's token must equal the oracle's: a strict position.
Otherwise the oracle's logit of the GPU's token must lie within the band of
its top-1: a near tie. The logit tolerance itself (err <= tol max|o|) is
checked separately. Without GPU logits (free-running calls) the band falls
back to 2 tol max|o|."""
import numpy as np

import oracle
from oracle import model as M

TOL = {"f32": 1e-3, "bf16": 2e-2}   # per-row relative logit tolerance


def rel_row_err(gpu, ref):
    """max_j |g_j - o_j| / max_j |o_j| for each row."""
    gpu = np.asarray(gpu, np.float64)
    ref = np.asarray(ref, np.float64)
    return np.abs(gpu - ref).max(-1) / np.abs(ref).max(-1)


def bands(ref_logits, gpu_logits=None, tol=None):
    """Per-row near-tie band: twice the row's measured logit error when the
    GPU's logits are given, else twice the tolerance times max|o|."""
    o = np.asarray(ref_logits, np.float64)
    if gpu_logits is not None:
        return 2.0 * np.abs(np.asarray(gpu_logits, np.float64) - o).max(-1)
    return 2.0 * tol * np.abs(o).max(-1)


def check_tokens(gpu_tok, ref_logits, tol=None, gpu_logits=None, min_strict=1):
    """Greedy agreement under teacher forcing (see the module docstring).
    Asserts at least min_strict strict positions; returns (strict, near)."""
    band = bands(ref_logits, gpu_logits, tol)
    strict = near = 0
    for g, o, b in zip(gpu_tok, ref_logits, band):
        o = np.asarray(o, np.float64)
        order = np.argsort(-o, kind="stable")
        top1, top2 = o[order[0]], o[order[1]]
        if top1 - top2 > b:
            assert int(g) == int(order[0]), (int(g), int(order[0]), top1 - top2, b)
            strict += 1
        else:
            near += 1
            assert o[int(g)] >= top1 - b, (int(g), o[int(g)], top1, b)
    assert strict >= min_strict, (strict, near)
    return strict, near


def check_free_run(gpu_tok, ref_tok, ref_logits, band, min_agree=1, along=None):
    """A free run (each side feeding its own choices back) against the
    oracle's: the tokens agree up to the first position where they differ;
    there the oracle's choice must have been a near tie (top-1 - top-2 within
    the band of that position) and the GPU's token must lie within the band
    of the top-1. Returns the number of leading tokens that agree (asserted
    to be at least min_agree, or the whole run).

    With `along` (a function that returns the oracle's logits at every
    position when the oracle is fed the GPU's own tokens), a run that
    leaves the oracle's at a near tie is followed to its end on the GPU's
    path: every later GPU token must be the oracle's choice on that path
    where the choice is clear, and lie within the band of its top-1 where it
    is a near tie (past the split, the band is the largest of `band`). The
    whole run is then checked, and the return value is its length."""
    gpu_tok = np.asarray(gpu_tok)
    ref_tok = np.asarray(ref_tok)
    n = min(gpu_tok.size, ref_tok.size)
    i = 0
    while i < n and int(gpu_tok[i]) == int(ref_tok[i]):
        i += 1
    if i < n:
        o = np.asarray(ref_logits[i], np.float64)
        top = np.sort(o)[-2:]
        assert top[1] - top[0] <= band[i], ("free run diverged at a clear position", i, top[1] - top[0], band[i])
        assert o[int(gpu_tok[i])] >= top[1] - band[i]
        if along is not None:
            lg = np.asarray(along(gpu_tok[:n]), np.float64)
            b = float(np.max(band))
            for j in range(i + 1, n):
                order = np.argsort(-lg[j], kind="stable")
                t1, t2, g = lg[j, order[0]], lg[j, order[1]], int(gpu_tok[j])
                if t1 - t2 > b:
                    assert g == int(order[0]), ("GPU path: not the oracle's clear choice", j, g, int(order[0]))
                else:
                    assert lg[j, g] >= t1 - b, ("GPU path: outside the near-tie band", j, g, t1 - lg[j, g], b)
            i = n
    assert i >= min(min_agree, n), (i, min_agree)
    return i


def check_ctc_entry(ctx, shape, b, seg, ref, tol, log=print):
    """CTC variant, batch entry b of the last encode pass against the oracle:
    head logits per frame within tol of the frame's largest magnitude; the
    device's per-frame ids equal the argmax of its own logits exactly; over
    the frames that cover the audio they equal the oracle's ids wherever the
    oracle's top-1 - top-2 margin exceeds twice the frame's measured logit
    error, and otherwise lie within that band. Returns (the device's ids of
    those frames, the number of near-tie frames)."""
    from oracle import ctc as OC
    from paper_2507_01021_amd import binding
    V = shape.n_vocab
    lg = ctx.debug_copy(binding.T_CTC_LOGITS, b, (1500, V))
    ids = ctx.debug_copy(binding.T_CTC_IDS, b, (1500,), np.int32)
    want = ref["logits"]
    err = (np.abs(lg - want).max(axis=1) / np.abs(want).max(axis=1)).max()
    log(f"entry {b}: logits rel err {err:.2e}")
    assert err < tol
    assert np.array_equal(ids, np.argmax(lg, axis=1))       # the device argmax is exact on its own logits
    T = OC.valid_frames(seg.audio.size)
    band = bands(want[:T], lg[:T])
    top2 = np.sort(want[:T], axis=1)[:, -2:]
    clear = (top2[:, 1] - top2[:, 0]) > band
    assert np.array_equal(ids[:T][clear], np.asarray(ref["ids"])[clear])
    for t in np.nonzero(~clear)[0]:
        assert want[t, ids[t]] >= want[t].max() - band[t]
    near = int((~clear).sum())
    log(f"entry {b}: {T} frames, {near} near ties, ids identical: {np.array_equal(ids[:T], np.asarray(ref['ids']))}")
    return ids[:T], near


def oracle_run(W, shape, segs, pad_mode=0, n_new=None, forced=None):
    """Features, encoder output, cross K/V and greedy tokens/logits of each
    segment, computed by the oracle one segment at a time."""
    out = []
    for s in segs:
        mel = oracle.log_mel_segment(s.audio, shape.n_mels, pad_mode)
        E = M.encoder(W, shape, mel[None])
        ckv = M._seg_ckv(M.cross_kv(W, shape, E), 0)
        n = s.max_new_tokens if n_new is None else n_new
        toks, lg = M.greedy(W, shape, ckv, s.prompt, n)
        out.append({"mel": mel, "E": E[0], "ckv": ckv, "tokens": toks, "logits": lg})
    return out


def float64_weights(W):
    """The same weights with the decoder's tensors already in float64, so the
    oracle's per-call conversion of them is a no-op (long decodes then take
    seconds per hundred steps instead of minutes). The values are unchanged."""
    import dataclasses
    return dataclasses.replace(W, values={k: np.asarray(v, np.float64) if k.startswith("dec.") else v
                                          for k, v in W.values.items()})


def drive_teacher_forced(ctx, slots, segs, ref, n_new):
    """Runs the GPU decode steps for `slots` (all encoded, same prompt
    length), feeding the oracle's tokens after the prompt. Returns per-slot
    lists of (argmax, logits) for the n_new generated positions."""
    n_prompt = len(segs[0].prompt)
    got_tok = [[] for _ in slots]
    got_lg = [[] for _ in slots]
    for step in range(n_prompt - 1 + n_new):
        gen_i = step - (n_prompt - 1)
        forced = None
        if gen_i >= 0:
            forced = [int(r["tokens"][gen_i]) for r in ref]
        tok, lg = ctx.decode_step(slots, forced=forced, logits=True)
        if gen_i < 0:
            assert np.all(tok == -1)
            continue
        for k in range(len(slots)):
            got_tok[k].append(int(tok[k]))
            got_lg[k].append(lg[k].copy())
    return got_tok, [np.stack(x) for x in got_lg]


def drain(ctx, slots):
    """Steps each listed slot until it is idle (generated all its tokens)."""
    from paper_2507_01021_amd import binding
    for s in slots:
        while True:
            try:
                ctx.decode_step([s])
            except binding.WhisperError as e:
                assert e.status == binding.E_STATE
                break
