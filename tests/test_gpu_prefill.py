"""One-shot prompt prefill (prefill = 1) through the C ABI: every encoded
segment's prompt positions 0..n_prompt-2 run through the decoder in one pass
at encode time, instead of one position per decode step.

Every decoder kernel treats its rows independently, so a prefilled slot's
caches, and therefore its logits and tokens, are bit-identical to those of
the same slot fed one prompt position per step. Checked on ragged prompts
of 1 to 100 tokens (161 prefill rows in one encoder pass: two chunks of at
most 128 rows), on the tiny fp32 model (also against the oracle, tolerance
as in test_gpu_parity) and on the bf16 base model, and in front of the
two-chain decode step of 40 bf16 slots."""
import sys

import numpy as np
import pytest

from paper_2507_01021_amd import binding, synth

from parity import TOL, bands, check_free_run, check_tokens, oracle_run, rel_row_err

pytestmark = pytest.mark.gpu

PROMPT_LENS = [1, 4, 60, 100]
N_NEW = 6


def log(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def ragged(shape, seed):
    """Four segments whose prompts are the standard prompt cut or extended
    with ordinary text ids to PROMPT_LENS tokens."""
    segs = synth.fixed_batch(shape, [16000, 48000, 112000, 480000], N_NEW, seed=seed)
    base = synth.prompt_for(shape)
    for s, n in zip(segs, PROMPT_LENS):
        s.prompt = (base + [400 + 37 * k % 9000 for k in range(n)])[:n]
    return segs


def step_logits(ctx, slots, segs, prefilled, forced_tokens):
    """Per slot: the logits of its N_NEW generated positions, the slot
    stepped alone, fed forced_tokens[k] after its prompt."""
    out = []
    for k, (slot, s) in enumerate(zip(slots, segs)):
        if not prefilled:
            for _ in range(len(s.prompt) - 1):
                tok = ctx.decode_step([slot])
                assert tok[0] == -1
        lg = []
        for j in range(N_NEW):
            _, l = ctx.decode_step([slot], forced=[int(forced_tokens[k][j])], logits=True)
            lg.append(l[0].copy())
        out.append(np.stack(lg))
    return out


@pytest.mark.parametrize("name", ["tiny", "base"])
def test_prefill_is_bit_identical_to_stepwise_prompt(name):
    shape = {"tiny": synth.TINY, "base": synth.BASE}[name]
    W = synth.make_weights(shape, 0)
    blob = synth.pack_blob(W)
    segs = ragged(shape, 21)
    slots = [0, 1, 2, 3]
    rows = sum(len(s.prompt) - 1 for s in segs)
    log(f"{name}: prompts {PROMPT_LENS}, {rows} prefill rows")
    forced = [[500 + 11 * j + k for j in range(N_NEW)] for k in range(len(segs))]
    res = {}
    for pf in (0, 1):
        with binding.Context(blob, max_slots=4, prefill=pf) as ctx:
            ctx.encode(segs, slots)
            lg = step_logits(ctx, slots, segs, pf == 1, forced)
            toks = [r["tokens"] for r in ctx.transcribe(segs)]
        res[pf] = (lg, toks)
    for k in range(len(segs)):
        assert np.array_equal(res[0][0][k], res[1][0][k]), (name, k)
        assert np.array_equal(res[0][1][k], res[1][1][k]), (name, k)
        log(f"{name} segment {k}: prompt {PROMPT_LENS[k]}, logits and tokens identical")


def test_prefill_matches_oracle_tiny():
    shape = synth.TINY
    W = synth.make_weights(shape, 0)
    segs = ragged(shape, 22)
    ref = oracle_run(W, shape, segs, n_new=N_NEW)
    with binding.Context(synth.pack_blob(W), max_slots=4, prefill=1) as ctx:
        ctx.encode(segs, [0, 1, 2, 3])
        lgs = step_logits(ctx, [0, 1, 2, 3], segs, True, [r["tokens"] for r in ref])
        got = ctx.transcribe(segs)
    for k, (r, g) in enumerate(zip(ref, got)):
        e = rel_row_err(lgs[k], r["logits"])
        log(f"tiny prefill segment {k}: prompt {PROMPT_LENS[k]}, logits rel err max {e.max():.2e}")
        assert e.max() < TOL["f32"]
        check_tokens(np.argmax(lgs[k], axis=-1), r["logits"], gpu_logits=lgs[k], min_strict=N_NEW // 2)
        check_free_run(g["tokens"], r["tokens"], r["logits"], bands(r["logits"], lgs[k]), min_agree=N_NEW // 2)


def test_prefill_bf16_two_chain_steps():
    """Prefill in front of the two-chain decode step (40 bf16 slots, chains
    of 16 and 24 rows) with ragged prompts of 1 to 9 tokens: the
    transcribed tokens equal those of prompts fed one position per step."""
    shape = synth.BASE.with_(n_enc=2, n_dec=2)
    W = synth.make_weights(shape, 0)
    blob = synth.pack_blob(W)
    segs = synth.uniform_batch(shape, 40, 5, seed=24)
    base = synth.prompt_for(shape)
    for k, sg in enumerate(segs):
        n = 1 + k % 9
        sg.prompt = (base + [300 + 13 * j for j in range(n)])[:n]
        sg.max_new_tokens = 4 + k % 5
    out = {}
    for pf in (0, 1):
        with binding.Context(blob, max_slots=40, prefill=pf) as ctx:
            log(f"base, 40 slots, prefill {pf}")
            out[pf] = [r["tokens"] for r in ctx.transcribe(segs)]
    for a, b in zip(out[0], out[1]):
        assert np.array_equal(a, b)


def test_prefill_with_refills():
    """The continuous batcher with prefill: more segments than slots, so
    slots are refilled while others decode; tokens equal prefill = 0's."""
    shape = synth.TINY
    W = synth.make_weights(shape, 0)
    blob = synth.pack_blob(W)
    segs = synth.fixed_batch(shape, [16000, 32000, 48000, 64000, 80000, 96000], 5, seed=23)
    for i, s in enumerate(segs):
        s.max_new_tokens = 3 + 2 * i
        s.prompt = s.prompt[: 1 + i % 4]
    out = {}
    for pf in (0, 1):
        with binding.Context(blob, max_slots=2, refill_min=1, prefill=pf) as ctx:
            out[pf] = [r["tokens"].tolist() for r in ctx.transcribe(segs)]
            st = ctx.stats()
        log(f"prefill {pf}: {st['decode_steps']} decode steps")
    assert out[0] == out[1]
