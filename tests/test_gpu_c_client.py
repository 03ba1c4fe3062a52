"""The C ABI from a plain C program (tests/c_client.c, compiled here with
the host C compiler against include/whisper_mi355x.h and the built
library): whisper_params_from_blob, whisper_ctx_create and one
whisper_batch_transcribe call, with no Python between the caller and the
library. Its output must equal the Python binding's call on the same
inputs token for token, echo every segment's user and segment id, and (on
the fp32 model) match the oracle's free run up to a near tie."""
import os
import shutil
import struct
import subprocess
import sys

import numpy as np
import pytest

from paper_2507_01021_amd import binding, synth

from parity import TOL, bands, check_free_run, oracle_run

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def log(*a):
    print(*a, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def client(tmp_path_factory):
    cc = shutil.which("gcc") or shutil.which("cc")
    if cc is None:
        pytest.skip("no host C compiler")
    out = str(tmp_path_factory.mktemp("c_client") / "whisper_c_client")
    lib_dir = os.path.dirname(binding.LIB_PATH)
    subprocess.run([cc, "-O2", "-std=c11", "-Wall", "-Werror", "-I", os.path.join(ROOT, "include"),
                    os.path.join(ROOT, "tests", "c_client.c"), "-L", lib_dir, "-lwhisper_mi355x",
                    f"-Wl,-rpath,{lib_dir}", "-o", out], check=True)
    return out


def write_segments(path, segs):
    with open(path, "wb") as f:
        f.write(struct.pack("<i", len(segs)))
        for s in segs:
            f.write(struct.pack("<iiiiq", s.audio.size, len(s.prompt), s.max_new_tokens, s.user_id, s.segment_id))
            f.write(np.asarray(s.prompt, np.int32).tobytes())
            f.write(np.asarray(s.audio, np.float32).tobytes())


def run_client(client, tmp_path, W, segs, slots):
    blob_path, seg_path = tmp_path / "w.blob", tmp_path / "segs.bin"
    synth.pack_blob(W).tofile(str(blob_path))
    write_segments(seg_path, segs)
    log(f"c client: {len(segs)} segments on {slots} slots")
    p = subprocess.run([client, str(blob_path), str(seg_path), str(slots)], stdout=subprocess.PIPE,
                       stderr=subprocess.PIPE, text=True, timeout=300)
    assert p.returncode == 0, p.stderr
    rows = [list(map(int, line.split())) for line in p.stdout.splitlines()]
    assert len(rows) == len(segs)
    return rows


def check_against_binding(rows, W, segs, slots):
    with binding.Context(synth.pack_blob(W), max_slots=slots) as ctx:
        want = ctx.transcribe(segs)
    for s, row, r in zip(segs, rows, want):
        sid, uid, status, n_tok, toks = row[0], row[1], row[2], row[3], np.array(row[4:], np.int32)
        assert (sid, uid, status) == (s.segment_id, s.user_id, 0)
        assert n_tok == s.max_new_tokens == toks.size
        assert np.array_equal(toks, r["tokens"])


def tagged(segs, first_id):
    for k, s in enumerate(segs):
        s.segment_id = first_id + 7919 * k
        s.user_id = 3 + k
    return segs


def test_c_client_tiny_matches_binding_and_oracle(client, tmp_path):
    shape, segs, slots = synth.workload("tiny-b2")
    W = synth.make_weights(shape, 0)
    segs = tagged(segs, 10 ** 12)
    rows = run_client(client, tmp_path, W, segs, slots)
    check_against_binding(rows, W, segs, slots)
    ref = oracle_run(W, shape, segs)
    for row, o in zip(rows, ref):
        check_free_run(np.array(row[4:]), o["tokens"], o["logits"], bands(o["logits"], tol=TOL["f32"]),
                       min_agree=4)


def test_c_client_base_bf16_with_refills(client, tmp_path):
    """Five ragged segments on three slots (two refills) in the bf16 model."""
    shape = synth.BASE
    W = synth.make_weights(shape, 0)
    segs = synth.uniform_batch(shape, 5, 12, seed=4)
    for k, s in enumerate(segs):
        s.max_new_tokens = 6 + 5 * k
    segs = tagged(segs, 5 * 10 ** 9)
    rows = run_client(client, tmp_path, W, segs, 3)
    check_against_binding(rows, W, segs, 3)
