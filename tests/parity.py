"""Shared parity helpers for the GPU tests: the tolerance rules for logits
and greedy tokens, and oracle runs on the same seeded inputs."""
import numpy as np

import oracle
from oracle import model as M

TOL = {"f32": 1e-3, "bf16": 2e-2}   # per-row relative logit tolerance


def rel_row_err(gpu, ref):
    """max_j |g_j - o_j| / max_j |o_j| for each row."""
    gpu = np.asarray(gpu, np.float64)
    ref = np.asarray(ref, np.float64)
    return np.abs(gpu - ref).max(-1) / np.abs(ref).max(-1)


def check_tokens(gpu_tok, ref_logits, tol):
    """Greedy agreement under teacher forcing: where the oracle's top-1 beats
    its top-2 by more than 2 tol max|o|, the GPU argmax must equal the
    oracle's; elsewhere the GPU token's oracle logit must lie within that
    band of the top-1. Returns the number of near-tie positions."""
    near = 0
    for g, o in zip(gpu_tok, ref_logits):
        o = np.asarray(o, np.float64)
        band = 2 * tol * np.abs(o).max()
        order = np.argsort(-o, kind="stable")
        top1, top2 = o[order[0]], o[order[1]]
        if top1 - top2 > band:
            assert int(g) == int(order[0]), (int(g), int(order[0]), top1 - top2, band)
        else:
            near += 1
            assert o[int(g)] >= top1 - band
    return near


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
