"""GPU parity at the full workload sizes, in the launch configuration the
benchmark uses (slots = the workload's slot count, encode passes of up to
32 segments), checked against the float64 oracle on sampled segments that
the oracle computes one by one: the encoder output of the sampled segments,
teacher-forced logits and greedy tokens of the first decode steps, and for
whole transcribe calls the exact id mapping and token placement of every
segment plus the sampled segments' leading tokens."""
import sys

import numpy as np
import pytest

from oracle import model as M
import oracle
from paper_2507_01021_amd import binding, synth

from parity import TOL, check_tokens, rel_row_err

pytestmark = pytest.mark.gpu


def log(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def oracle_segment(W, shape, seg, n_steps):
    mel = oracle.log_mel_segment(seg.audio, shape.n_mels)
    E = M.encoder(W, shape, mel[None])
    ckv = M._seg_ckv(M.cross_kv(W, shape, E), 0)
    toks, lg = M.greedy(W, shape, ckv, seg.prompt, n_steps)
    return E[0], toks, lg


def first_near_tie(tokens_ref, logits_ref, tol):
    """Index of the first position whose top-1/top-2 margin is within the
    tie band (a free run may legitimately diverge after it)."""
    for i, o in enumerate(logits_ref):
        band = 2 * tol * np.abs(o).max()
        top = np.sort(o)[-2:]
        if top[1] - top[0] <= band:
            return i
    return len(tokens_ref)


def run_teacher_forced(ctx, slots, k, ref_toks, n_prompt, n_gen, other_tok=220):
    """Steps every listed slot; slot index k is forced with the oracle's
    tokens, the others with a fixed token (they are independent)."""
    toks, lgs = [], []
    for step in range(n_prompt - 1 + n_gen):
        g = step - (n_prompt - 1)
        forced = None
        if g >= 0:
            forced = [other_tok] * len(slots)
            forced[k] = int(ref_toks[g])
        tok, lg = ctx.decode_step(slots, forced=forced, logits=True)
        if g >= 0:
            toks.append(int(tok[k]))
            lgs.append(lg[k].astype(np.float64))
    return toks, np.stack(lgs)


def drain_all(ctx, slots):
    """Steps slots that were encoded together with equal lengths until they
    all become idle at once."""
    while True:
        try:
            ctx.decode_step(slots)
        except binding.WhisperError as e:
            assert e.status == binding.E_STATE
            return


@pytest.mark.parametrize("name,sample", [("base-b16", [3]), ("large-v3-b32", [17])])
def test_fixed_batch_bench_config(name, sample):
    shape, segs, slots = synth.workload(name)
    log(f"{name}: weights")
    W = synth.make_weights(shape, 0)
    with binding.Context(synth.pack_blob(W), max_slots=slots, max_encode_batch=min(slots, 32)) as ctx:
        log(f"{name}: encode {len(segs)} segments")
        ctx.encode(segs, list(range(len(segs))))
        n_gen = 4
        refs = {}
        for k in sample:
            E_ref, toks_ref, lg_ref = refs[k] = oracle_segment(W, shape, segs[k], n_gen)
            E = ctx.debug_copy(binding.T_ENC_OUT, k, (1500, shape.d))
            e = rel_row_err(E, E_ref).max()
            log(f"{name}: segment {k} encoder rel err {e:.3e}")
            assert e < TOL["bf16"]
            toks, lgs = run_teacher_forced(ctx, list(range(len(segs))), k, toks_ref, len(segs[k].prompt), n_gen)
            e = rel_row_err(lgs, lg_ref).max()
            log(f"{name}: segment {k} teacher-forced logits rel err {e:.3e}")
            assert e < TOL["bf16"]
            check_tokens(toks, lg_ref, TOL["bf16"])
        drain_all(ctx, list(range(len(segs))))
        log(f"{name}: transcribe")
        res = ctx.transcribe(segs)
        for s, r in zip(segs, res):
            assert (r["user_id"], r["segment_id"], r["status"]) == (s.user_id, s.segment_id, 0)
            assert r["tokens"].size == s.max_new_tokens
        for k in sample:
            _, toks_ref, lg_ref = refs[k]
            upto = first_near_tie(toks_ref, lg_ref, TOL["bf16"])
            assert np.array_equal(res[k]["tokens"][:upto], toks_ref[:upto])


@pytest.mark.parametrize("name,sample", [("small-u8-b64", [5, 40]), ("turbo-u64-q512", [300])])
def test_continuous_batching_workload(name, sample):
    """Ragged lengths and slot refill: every segment's tokens land at its
    input-order offset, and sampled segments' leading tokens equal the
    oracle's solo greedy run."""
    shape, segs, slots = synth.workload(name)
    log(f"{name}: weights")
    W = synth.make_weights(shape, 0)
    with binding.Context(synth.pack_blob(W), max_slots=slots, max_encode_batch=min(slots, 32)) as ctx:
        log(f"{name}: transcribe {len(segs)} segments with {slots} slots")
        ctx.stats(reset=True)
        res = ctx.transcribe(segs)
        st = ctx.stats()
        # work counters are exact: every segment takes n_prompt - 1 + max_new steps,
        # attending 1, 2, ... positions
        steps = [len(s.prompt) - 1 + s.max_new_tokens for s in segs]
        assert st["segments_encoded"] == len(segs)
        assert st["rows_decoded"] == sum(steps)
        assert st["positions_attended"] == sum(k * (k + 1) // 2 for k in steps)
        assert max(steps) <= st["decode_steps"] <= sum(steps)
        assert st["refill_batches"] >= -(-len(segs) // min(slots, 32))
        for s, r in zip(segs, res):
            assert (r["user_id"], r["segment_id"], r["status"]) == (s.user_id, s.segment_id, 0)
            assert r["tokens"].size == s.max_new_tokens
            assert np.all((r["tokens"] >= 0) & (r["tokens"] < shape.n_vocab))
        for k in sample:
            n_gen = min(4, segs[k].max_new_tokens)
            _, toks_ref, lg_ref = oracle_segment(W, shape, segs[k], n_gen)
            upto = first_near_tie(toks_ref, lg_ref, TOL["bf16"])
            log(f"{name}: segment {k} oracle tokens {toks_ref.tolist()} gpu {res[k]['tokens'][:n_gen].tolist()}")
            assert np.array_equal(res[k]["tokens"][:upto], toks_ref[:upto])
        # the same segment alone gives the same tokens (batch invariance)
        k = sample[0]
        solo = ctx.transcribe([segs[k]])[0]
        assert np.array_equal(solo["tokens"], res[k]["tokens"])
