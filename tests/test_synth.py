"""Seeded generators: determinism, value distributions, blob layout and the
workload recipes (segment lengths 3-30 s, Poisson arrivals per user)."""
import struct

import numpy as np

from paper_2507_01021_amd import synth


def test_weights_deterministic_and_distributed():
    s = synth.TINY.with_(d=64, n_head=1, n_enc=1, n_dec=1, n_vocab=300)
    a, b = synth.make_weights(s, 0), synth.make_weights(s, 0, threads=1)
    c = synth.make_weights(s, 1)
    for k in a.values:
        assert np.array_equal(a[k], b[k])
    assert not np.array_equal(a["dec.tok_emb"], c["dec.tok_emb"])
    w = a["enc.0.mlp.fc1.w"]
    assert abs(w.mean()) < 2e-3 and abs(w.std() - 0.02) < 1e-3
    g = a["enc.0.attn_ln.g"]
    assert abs(g.mean() - 1.0) < 0.01


def test_bf16_rounding_nearest_even():
    x = np.array([1.0, 1.0 + 2 ** -8, 1.0 + 3 * 2 ** -9, -2.5, 3.0e-3], dtype=np.float32)
    r = synth.bf16_to_f32(synth.round_to_bf16(x))
    assert r[0] == 1.0
    assert r[1] == 1.0                    # halfway, ties to even (mantissa 0)
    assert r[2] == 1.0 + 2 ** -7          # halfway, ties to even (rounds up)
    assert r[3] == -2.5
    assert abs(r[4] - 3.0e-3) <= 3.0e-3 * 2 ** -8
    s = synth.BASE.with_(d=64, n_head=1, n_enc=1, n_dec=1, n_vocab=300)
    w = synth.make_weights(s, 0)
    for k, v in w.values.items():
        assert np.array_equal(synth.bf16_to_f32(w.bits[k]), v)


def test_blob_layout():
    for s in (synth.TINY.with_(n_vocab=500), synth.BASE.with_(n_vocab=500, n_enc=1, n_dec=1)):
        w = synth.make_weights(s, 0)
        blob = synth.pack_blob(w)
        lay, total = synth.blob_layout(s)
        assert blob.size == total and total % 256 == 0
        hdr = struct.unpack("<8s14i", blob[:64].tobytes())
        assert hdr[0] == b"WHSPMI01" and hdr[1] == 1 and hdr[2] == (0 if s.dtype == "f32" else 1)
        assert hdr[3:14] == (s.n_mels, 1500, s.d, s.n_head, s.n_enc, s.n_vocab, 448, s.d,
                             s.n_head, s.n_dec, len(lay))
        esz = 4 if s.dtype == "f32" else 2
        for name, shp, off in lay:
            assert off % 256 == 0
            raw = blob[off: off + int(np.prod(shp)) * esz]
            if s.dtype == "f32":
                assert np.array_equal(raw.view(np.float32).reshape(shp), w[name])
            else:
                assert np.array_equal(synth.bf16_to_f32(raw.view(np.uint16)).reshape(shp), w[name])


def test_workload_recipes():
    s, segs, slots = synth.workload("tiny-b2")
    assert [x.audio.size for x in segs] == [48000, 112000] and slots == 2
    assert all(x.max_new_tokens == 16 and x.prompt == [50258, 50259, 50359, 50363] for x in segs)
    s, segs, slots = synth.workload("base-b16")
    assert len(segs) == 16 and all(48000 <= x.audio.size <= 480000 for x in segs)
    s, segs, slots = synth.workload("small-u8-b64")
    assert len(segs) == 64 and len({x.user_id for x in segs}) == 8
    arr = [x.arrival_us for x in segs]
    assert arr == sorted(arr)
    assert all(16 <= x.max_new_tokens <= 128 for x in segs)
    assert len({x.segment_id for x in segs}) == 64
    a = segs[0].audio
    assert a.dtype == np.float32 and 0.05 < a.std() < 0.4


def test_poisson_gaps():
    segs = synth.poisson_users(synth.TINY, 1, 400, 5.0, 1, 1, seed=9)
    gaps = np.diff([0] + [x.arrival_us for x in segs]) / 1e6
    assert abs(gaps.mean() - 5.0) < 0.6 and abs(gaps.std() - 5.0) < 0.8
