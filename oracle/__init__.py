"""CPU oracle for batched Whisper inference over independent speech segments.

TEST INFRASTRUCTURE ONLY. Only the test suite, the package smoke check and
the benchmark's CPU-baseline leg may import or call anything here; the
product (the HIP library and its Python binding) never does, and shares no
code with it.

The oracle is a plain, slow, float64 NumPy implementation of what the
method computes (Section 2.3 and Listing 1 of the paper): per-segment log-mel
features padded to a 30 s window, stacked into a batch, encoded, then
decoded greedily from a prompt ending in the no-timestamps token. Segments
are independent units, so batching changes speed, not results.

The paper fixes neither the network nor the front end; both follow the
public Whisper architecture (pre-LN transformer encoder-decoder, conv stem,
sinusoidal encoder positions, learned decoder positions, tied output head)
and its log-mel recipe; both sides of every comparison use the same readings.

The CTC variant (oracle/ctc.py) reads the paper's remark on encoder-only
CTC recognisers as the same encoder with a linear head and greedy best-path
decoding.

Pins (tests/test_oracle_*.py): DFT vs numpy.fft, a bin-centred tone's closed
form, Parseval, Slaney mel closed forms and a library filter bank, the whole
front end and the whole network against an independent library
implementation (transformers' Whisper) on CPU, softmax and layer-norm
invariants, causal mask vs brute force, cached decode vs full recompute,
batch vs solo, and argmax tie-breaking.
"""
from .frontend import (hann_periodic, frame_audio, power_spectrum, hz_to_mel, mel_to_hz,
                       mel_filterbank, log_mel, log_mel_segment)
from .model import (layer_norm, gelu, softmax, mha, conv_stem, sinusoid_pe, encoder,
                    cross_kv, decoder_logits_full, DecoderCache, decoder_step, greedy,
                    transcribe, transcribe_batch)
from .ctc import valid_frames, ctc_logits, best_path, collapse, transcribe_ctc

__all__ = [
    "hann_periodic", "frame_audio", "power_spectrum", "hz_to_mel", "mel_to_hz",
    "mel_filterbank", "log_mel", "log_mel_segment", "layer_norm", "gelu", "softmax",
    "mha", "conv_stem", "sinusoid_pe", "encoder", "cross_kv", "decoder_logits_full",
    "DecoderCache", "decoder_step", "greedy", "transcribe", "transcribe_batch",
]
