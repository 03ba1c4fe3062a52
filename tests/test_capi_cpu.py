"""Host-side checks of the C-ABI library (no GPU needed): it loads, exports
every function the header declares, parses weight blobs, and rejects bad
arguments before touching a device."""
import ctypes as C
import os
import re

import numpy as np
import pytest

from paper_2507_01021_amd import binding, synth

HEADER = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "include",
                      "whisper_mi355x.h")


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(binding.LIB_PATH):
        pytest.skip("library not built (python -m paper_2507_01021_amd.build)")
    return binding.load()


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(whisper_[a-z_]+)\s*\(", text)))


def test_header_declarations_match_binding():
    assert declared_functions() == sorted(binding.EXPORTS)


def test_library_exports_every_declared_symbol(lib):
    for name in declared_functions():
        assert hasattr(lib, name), name


def test_struct_layouts_match_header(tmp_path):
    """The ctypes mirrors have the sizes and offsets a C compiler gives the
    header's structs."""
    fields = {"whisper_params": [f for f, _ in binding.whisper_params._fields_],
              "whisper_segment": [f for f, _ in binding.whisper_segment._fields_],
              "whisper_result": [f for f, _ in binding.whisper_result._fields_],
              "whisper_stats": [f for f, _ in binding.whisper_stats._fields_]}
    lines = ['#include <stdio.h>', '#include <stddef.h>', f'#include "{HEADER}"', "int main(void) {"]
    for st, fs in fields.items():
        lines.append(f'printf("{st} %zu\\n", sizeof({st}));')
        for f in fs:
            lines.append(f'printf("{st}.{f} %zu\\n", offsetof({st}, {f}));')
    lines.append("return 0; }")
    src = tmp_path / "layout.c"
    src.write_text("\n".join(lines))
    exe = tmp_path / "layout"
    import subprocess
    subprocess.run(["gcc", "-o", str(exe), str(src)], check=True)
    got = dict(l.split() for l in subprocess.run([str(exe)], capture_output=True, text=True,
                                                  check=True).stdout.splitlines())
    for st, fs in fields.items():
        cls = getattr(binding, st)
        assert int(got[st]) == C.sizeof(cls), st
        for f in fs:
            assert int(got[f"{st}.{f}"]) == getattr(cls, f).offset, (st, f)


def test_params_from_blob(lib):
    s = synth.TINY.with_(n_vocab=300, n_enc=1, n_dec=1)
    blob = synth.pack_blob(synth.make_weights(s, 0))
    p = binding.params_from_blob(blob)
    assert (p.n_mels, p.n_audio_state, p.n_audio_head, p.n_audio_layer, p.n_vocab, p.n_text_layer,
            p.dtype, p.max_slots) == (80, 384, 6, 1, 300, 1, 0, 32)
    bad = blob.copy()
    bad[0] = ord("X")
    with pytest.raises(binding.WhisperError) as e:
        binding.params_from_blob(bad)
    assert e.value.status == binding.E_FORMAT


@pytest.mark.parametrize("field,value", [("max_slots", 0), ("max_slots", 129), ("pad_mode", 2),
                                         ("max_encode_batch", 99), ("refill_min", -1), ("prefill", 2)])
def test_create_rejects_bad_params_before_device(lib, field, value):
    s = synth.TINY.with_(n_vocab=300, n_enc=1, n_dec=1)
    blob = synth.pack_blob(synth.make_weights(s, 0))
    p = binding.params_from_blob(blob)
    setattr(p, field, value)
    h = C.c_void_p()
    st = lib.whisper_ctx_create(C.byref(p), blob.ctypes.data, blob.nbytes, 0, C.byref(h))
    assert st == binding.E_INVAL and not h.value
    assert lib.whisper_last_error(None)


def test_create_rejects_params_not_matching_blob(lib):
    s = synth.TINY.with_(n_vocab=300, n_enc=1, n_dec=1)
    blob = synth.pack_blob(synth.make_weights(s, 0))
    p = binding.params_from_blob(blob)
    p.n_vocab = 301
    h = C.c_void_p()
    assert lib.whisper_ctx_create(C.byref(p), blob.ctypes.data, blob.nbytes, 0, C.byref(h)) == binding.E_FORMAT


def test_null_context_calls_fail_cleanly(lib):
    assert lib.whisper_batch_encode(None, None, 1, None) == binding.E_INVAL
    assert lib.whisper_batch_decode_step(None, None, 1, None, None, None) == binding.E_INVAL
    assert lib.whisper_batch_transcribe(None, None, 1, None, 0, None) == binding.E_INVAL
    st = binding.whisper_stats()
    assert lib.whisper_stats_read(None, C.byref(st), 0) == binding.E_INVAL
    us = C.c_double()
    assert lib.whisper_time_kernel(None, binding.K_CROSS_ATTN, 1, 1, C.byref(us)) == binding.E_INVAL
    lib.whisper_ctx_destroy(None)


def test_params_from_ctc_blob(lib):
    """An encoder-only CTC blob (n_text_layer 0) parses; its layout ends with the head."""
    shape = synth.CTC_TINY
    lay, total = synth.blob_layout(shape)
    assert [n for n, _, _ in lay][-2:] == ["ctc.w", "ctc.b"]
    blob = np.zeros(total, dtype=np.uint8)
    w = synth.make_weights(shape.with_(n_enc=1), 0)
    hdr = synth.pack_blob(w)[:256]
    p = binding.whisper_params()
    assert lib.whisper_params_from_blob(hdr.ctypes.data, hdr.size, C.byref(p)) == 0
    assert (p.n_text_layer, p.n_vocab, p.n_audio_layer) == (0, 256, 1)


def test_prefill_rejected_for_ctc_models(lib):
    """prefill = 1 needs a decoder: a CTC blob's context is refused before any device work."""
    shape = synth.CTC_TINY.with_(n_enc=1)
    lay, total = synth.blob_layout(shape)
    blob = np.zeros(total, dtype=np.uint8)
    blob[:256] = synth.pack_blob(synth.make_weights(shape, 0))[:256]
    p = binding.params_from_blob(blob)
    p.prefill = 1
    h = C.c_void_p()
    st = lib.whisper_ctx_create(C.byref(p), blob.ctypes.data, blob.nbytes, 0, C.byref(h))
    assert st == binding.E_INVAL and not h.value
    assert b"prefill" in lib.whisper_last_error(None)


def test_greedy_keys_on_host(lib):
    """The decode step's greedy-choice keys, run on the host: the largest
    logit wins, the lowest id among equal logits, negative values and -inf
    order correctly, excluded ids are skipped, and a row with every id
    excluded yields token 0 with its flag raised (the step's error); a row of
    -inf logits yields id 0 without an error."""
    V = 70
    rng = np.random.default_rng(3)
    lg = rng.normal(size=(6, V)).astype(np.float32)
    lg[1, 5] = lg[1, 40] = lg[1].max() + 1.0           # tie: the lower id
    lg[2] = -np.abs(lg[2]) - 1.0                        # all negative
    lg[2, 66] = -0.5
    lg[3] = -np.inf
    lg[3, 69] = -1e30                                   # the only finite value
    lg[4, 33] = 1e30
    tok, bad = binding.test_greedy_keys(lg)
    assert tok.tolist() == [int(np.argmax(r)) for r in lg]
    assert tok[1] == 5 and tok[2] == 66 and tok[3] == 69 and not bad.any()
    tok, bad = binding.test_greedy_keys(lg, excluded_ids=[33, 5])
    assert tok[4] != 33 and tok[1] == 40 and not bad.any()
    tok, bad = binding.test_greedy_keys(lg[:1], excluded_ids=range(V))
    assert tok.tolist() == [0] and bad.tolist() == [1]
    # every logit -inf: still a defined choice, the first maximum (id 0), as argmax gives
    tok, bad = binding.test_greedy_keys(np.full((2, V), -np.inf, np.float32))
    assert tok.tolist() == [0, 0] and not bad.any()


def test_cross_cache_layer_index_is_exact():
    """The cross-attention K/V epilogues find the layer of a stacked weight
    column n as trunc((n + 1/2) * fp32(1/d)) in fp32 arithmetic instead of an
    integer division. The bound behind it (n < 2^20, d <= 2^11) covers every
    width the library accepts (64 x 6 .. 64 x 32) with up to 256 decoder
    layers; checked here exhaustively in the same fp32 arithmetic."""
    for d in (384, 512, 768, 1024, 1280, 1536, 2048):
        n = np.arange(256 * d, dtype=np.int64)
        rd = np.float32(1.0) / np.float32(d)
        l = ((n.astype(np.float32) + np.float32(0.5)) * rd).astype(np.int64)
        assert np.array_equal(l, n // d), d


def test_c_client_builds_against_the_header(lib, tmp_path):
    """tests/c_client.c (the plain C caller the GPU tests run) compiles
    warning-free against the header, links the library and rejects a
    missing argument before any library call."""
    import shutil
    import subprocess
    cc = shutil.which("gcc") or shutil.which("cc")
    if cc is None:
        pytest.skip("no host C compiler")
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    lib_dir = os.path.dirname(binding.LIB_PATH)
    exe = str(tmp_path / "whisper_c_client")
    subprocess.run([cc, "-O2", "-std=c11", "-Wall", "-Wextra", "-Werror", "-I", os.path.join(root, "include"),
                    os.path.join(root, "tests", "c_client.c"), "-L", lib_dir, "-lwhisper_mi355x",
                    f"-Wl,-rpath,{lib_dir}", "-o", exe], check=True)
    p = subprocess.run([exe], capture_output=True, text=True, timeout=60)
    assert p.returncode == 1 and "usage" in p.stderr
