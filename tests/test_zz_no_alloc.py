"""The allocation-free decode step (whisper_batch_decode_step_noalloc)
against the regular one (whisper_batch_decode_step), through the C ABI:
two contexts with the same weights and segments, one stepped by each entry
point; the greedy tokens of every step must be identical (integer output,
bit-exact), over two calls in a row where the second steps fewer slots,
and the slots' state must advance the same way."""
import sys

import numpy as np
import pytest

from paper_2507_01021_amd import binding, synth

pytestmark = pytest.mark.gpu


def log(*a):
    print(*a, flush=True)
    sys.stdout.flush()


@pytest.mark.parametrize("shape_name,n_seg", [("base", 16), ("tiny", 2)])
def test_noalloc_step_matches_regular_step(shape_name, n_seg):
    import torch
    shape = synth.SHAPES[shape_name]
    W = synth.make_weights(shape, 0)
    blob = synth.pack_blob(W)
    segs = synth.uniform_batch(shape, n_seg, 12, seed=7)
    slots = list(range(n_seg))
    small = slots[: max(1, n_seg // 2)]
    out = torch.full((n_seg,), -7, dtype=torch.int32, device="cuda:0")
    with binding.Context(blob, max_slots=n_seg) as ref, binding.Context(blob, max_slots=n_seg) as na:
        log(f"{shape_name}: encode {n_seg} segments in both contexts")
        ref.encode(segs, slots)
        na.encode(segs, slots)
        # call 1: every slot, through the prompt and into generation; call 2: fewer slots
        for rows in (slots, small):
            for step in range(4):
                want = ref.decode_step(rows)
                out.fill_(-7)
                na.decode_step_noalloc(rows, out.data_ptr())
                torch.cuda.synchronize()
                got = out[: len(rows)].cpu().numpy()
                log(f"{shape_name}: {len(rows)} rows, step {step}: {got.tolist()[:6]}")
                assert np.array_equal(got, want)
                assert np.all(out[len(rows):].cpu().numpy() == -7)      # nothing written past n
        for s in slots:
            assert np.array_equal(na.slot_tokens(s), ref.slot_tokens(s))
        # without an output buffer the step still runs and advances the slots
        na.decode_step_noalloc(small)
        ref.decode_step(small)
        torch.cuda.synchronize()
        for s in small:
            assert np.array_equal(na.slot_tokens(s), ref.slot_tokens(s))


def test_noalloc_step_rejects_sizes_beyond_the_array():
    shape = synth.TINY
    W = synth.make_weights(shape, 0)
    segs = synth.uniform_batch(shape, 2, 4, seed=8)
    with binding.Context(synth.pack_blob(W), max_slots=128, max_encode_batch=2) as ctx:
        ctx.encode(segs, [0, 1])
        with pytest.raises(binding.WhisperError) as e:
            ctx.decode_step_noalloc(list(range(65)))               # above the row limit
        assert e.value.status == binding.E_CAPACITY
        # fp32 logits of 64 rows x 51865 ids do not fit the array
        many = [synth.uniform_batch(shape, 1, 4, seed=9)[0] for _ in range(40)]
        ctx.encode(many, list(range(2, 42)))
        with pytest.raises(binding.WhisperError) as e:
            ctx.decode_step_noalloc(list(range(42)))
        assert e.value.status == binding.E_CAPACITY and "bytes of scratch" in str(e.value)
        ctx.decode_step_noalloc([0, 1])                           # a size that fits still works
