"""Decode steps of 32 or more bf16 rows run as two chains on two streams;
while the slot list is unchanged the chains are not joined between steps.
A row's result never depends on the other rows or on the stream timing, so
every token equals the per-step-join run's (WHISPER_FREE_CHAINS=0, read
when a context is created)."""
import os
import sys

import numpy as np
import pytest

from paper_2507_01021_amd import binding, synth

pytestmark = pytest.mark.gpu


def test_chains_apart_equal_joined():
    shape = synth.BASE
    W = synth.make_weights(shape, 0)
    blob = synth.pack_blob(W)
    segs = synth.fixed_batch(shape, [16000 * (3 + i % 27) for i in range(40)], 12, seed=31)
    for i, s in enumerate(segs):
        # 34 long segments keep an unchanged list of >= 32 rows for ~20 steps;
        # the short ones retire early and change the list meanwhile
        s.max_new_tokens = 24 if i < 34 else 4 + i % 5
    out = {}
    for mode in ("apart", "joined"):
        if mode == "joined":
            os.environ["WHISPER_FREE_CHAINS"] = "0"
        try:
            with binding.Context(blob, max_slots=40, refill_min=8) as ctx:
                out[mode] = [r["tokens"].tolist() for r in ctx.transcribe(segs)]
        finally:
            os.environ.pop("WHISPER_FREE_CHAINS", None)
        print(f"{mode}: {sum(len(t) for t in out[mode])} tokens", flush=True)
        sys.stdout.flush()
    assert out["apart"] == out["joined"]
    assert all(len(t) == s.max_new_tokens for t, s in zip(out["apart"], segs))


def test_stamped_cross_attention_steps():
    """Cross-attention spans stamped inside the captured split steps
    (WHISPER_K_CROSS_ATTN_STEP): the tokens equal an unstamped call's, every
    launch (chain x layer x step) is counted, and the average span is
    positive and below 5 ms."""
    shape = synth.BASE
    W = synth.make_weights(shape, 0)
    segs = synth.uniform_batch(shape, 40, 6, seed=32)
    with binding.Context(synth.pack_blob(W), max_slots=40) as ctx:
        want = [r["tokens"].tolist() for r in ctx.transcribe(segs)]
        ctx.stats(reset=True)
        ctx.profile_enable(binding.K_CROSS_ATTN_STEP, True)
        got = [r["tokens"].tolist() for r in ctx.transcribe(segs)]
        ms, n = ctx.profile_read(binding.K_CROSS_ATTN_STEP)
        ctx.profile_enable(binding.K_CROSS_ATTN_STEP, False)
        st = ctx.stats()
    print(f"stamped: {n} launches, {ms * 1e3 / max(n, 1):.2f} us each", flush=True)
    assert got == want
    steps = st["decode_steps"]
    # one launch per chain and layer: two chains in steps of 32 or more rows, else one
    assert steps > 0 and n % shape.n_dec == 0 and shape.n_dec * steps <= n <= 2 * shape.n_dec * steps
    assert 0 < ms / n < 5.0
