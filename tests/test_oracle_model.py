"""Pins for the oracle network: attention, layer norm, GELU, conv stem,
positional tables, the whole encoder-decoder against an independent library
implementation (transformers' Whisper, float64, CPU), cached decoding
against full recompute, batch against solo runs, and greedy tie-breaking."""
import math

import numpy as np
import pytest
import torch

import oracle
from oracle import model as M
from paper_2507_01021_amd import synth

SMALL_SHAPE = synth.TINY.with_(name="pin", d=128, n_head=2, n_enc=2, n_dec=2, n_vocab=1000)
PROMPT = [1, 2, 3, 4]


def _rng(seed=0):
    return np.random.Generator(np.random.PCG64(seed))


@pytest.fixture(scope="module")
def weights():
    return synth.make_weights(SMALL_SHAPE, seed=0)


@pytest.fixture(scope="module")
def segments():
    segs = synth.fixed_batch(SMALL_SHAPE, [48000, 23456], 6, seed=1)
    for s in segs:
        s.prompt = list(PROMPT)
    return segs


# ---------------------------------------------------------------- primitives

def test_softmax_rows_sum_to_one():
    s = _rng(1).standard_normal((4, 9, 17)) * 30
    p = M.softmax(s)
    assert np.allclose(p.sum(-1), 1.0, atol=1e-14)
    assert np.all(p >= 0)


def test_attention_identical_keys_gives_mean_value():
    q = _rng(2).standard_normal((3, 5, 64))
    k = np.broadcast_to(_rng(3).standard_normal(64), (3, 11, 64))
    v = _rng(4).standard_normal((3, 11, 64))
    assert np.allclose(M.attention(q, k, v), v.mean(1, keepdims=True).repeat(5, 1), atol=1e-14)


@pytest.mark.parametrize("causal", [False, True])
def test_attention_matches_torch_sdpa(causal):
    g = _rng(5)
    q, k, v = (g.standard_normal((2, 3, 7, 64)) for _ in range(3))
    want = torch.nn.functional.scaled_dot_product_attention(
        torch.from_numpy(q), torch.from_numpy(k), torch.from_numpy(v), is_causal=causal).numpy()
    assert np.allclose(M.attention(q, k, v, causal), want, atol=1e-12)


def test_causal_mask_matches_per_prefix_bruteforce():
    g = _rng(6)
    for t in range(1, 9):
        q, k, v = (g.standard_normal((t, 64)) for _ in range(3))
        got = M.attention(q, k, v, causal=True)
        for i in range(t):
            s = np.array([sum(q[i, c] * k[j, c] for c in range(64)) / 8.0 for j in range(i + 1)])
            e = np.exp(s - s.max())
            want = (e / e.sum()) @ v[: i + 1]
            assert np.allclose(got[i], want, atol=1e-12)


def test_layer_norm_standardises():
    x = _rng(7).standard_normal((6, 384)) * 3 + 5
    y = M.layer_norm(x, np.ones(384), np.zeros(384))
    assert np.allclose(y.mean(-1), 0.0, atol=1e-12)
    var = x.var(-1)
    assert np.allclose(y.var(-1), var / (var + 1e-5), atol=1e-12)
    want = torch.nn.functional.layer_norm(torch.from_numpy(x), (384,), eps=1e-5).numpy()
    assert np.allclose(y, want, atol=1e-12)


def test_gelu_is_erf_form():
    x = np.linspace(-6, 6, 1001)
    want = torch.nn.functional.gelu(torch.from_numpy(x), approximate="none").numpy()
    assert np.allclose(M.gelu(x), want, atol=1e-15)
    tanh_form = torch.nn.functional.gelu(torch.from_numpy(x), approximate="tanh").numpy()
    assert np.abs(M.gelu(x) - tanh_form).max() > 1e-4     # the two forms are distinguishable


def test_conv_stem_matches_bruteforce_and_torch():
    g = _rng(8)
    cin, cout, t = 3, 4, 10
    x = g.standard_normal((1, cin, t))
    w1, b1 = g.standard_normal((cout, cin, 3)), g.standard_normal(cout)
    for stride in (1, 2):
        got = M._conv1d(x, w1, b1, stride)
        t_out = (t - 1) // stride + 1
        assert got.shape == (1, cout, t_out)
        for o in range(cout):
            for j in range(t_out):
                acc = b1[o]
                for c in range(cin):
                    for tap in range(3):
                        src = stride * j + tap - 1
                        if 0 <= src < t:
                            acc += w1[o, c, tap] * x[0, c, src]
                assert abs(got[0, o, j] - acc) < 1e-12
        want = torch.nn.functional.conv1d(torch.from_numpy(x), torch.from_numpy(w1),
                                          torch.from_numpy(b1), stride=stride, padding=1).numpy()
        assert np.allclose(got, want, atol=1e-12)


def test_sinusoid_table():
    pe = M.sinusoid_pe(1500, 384)
    assert np.array_equal(pe[0], np.concatenate([np.zeros(192), np.ones(192)]))
    # the slowest channel has timescale 10000: angle t * 1e-4
    assert np.allclose(pe[:, 191], np.sin(np.arange(1500) * 1e-4), atol=1e-15)
    assert np.allclose(pe[:, 0], np.sin(np.arange(1500)), atol=1e-12)
    tfm = pytest.importorskip("transformers.models.whisper.modeling_whisper")
    prev = torch.get_default_dtype()
    torch.set_default_dtype(torch.float64)
    try:
        lib = tfm.sinusoids(1500, 384).numpy()
    finally:
        torch.set_default_dtype(prev)
    assert np.allclose(pe, lib, atol=1e-12)


# ------------------------------------------------ whole network vs a library

def _hf_model(shape, W):
    tf = pytest.importorskip("transformers")
    tfm = pytest.importorskip("transformers.models.whisper.modeling_whisper")
    cfg = tf.WhisperConfig(
        vocab_size=shape.n_vocab, num_mel_bins=shape.n_mels, encoder_layers=shape.n_enc,
        decoder_layers=shape.n_dec, encoder_attention_heads=shape.n_head,
        decoder_attention_heads=shape.n_head, d_model=shape.d, encoder_ffn_dim=4 * shape.d,
        decoder_ffn_dim=4 * shape.d, max_source_positions=1500, max_target_positions=448,
        activation_function="gelu", pad_token_id=0, bos_token_id=1, eos_token_id=2,
        decoder_start_token_id=1, dropout=0.0, attention_dropout=0.0, activation_dropout=0.0)
    m = tf.WhisperForConditionalGeneration(cfg).double().eval()
    sd = {"model.encoder.conv1.weight": W["enc.conv1.w"], "model.encoder.conv1.bias": W["enc.conv1.b"],
          "model.encoder.conv2.weight": W["enc.conv2.w"], "model.encoder.conv2.bias": W["enc.conv2.b"],
          "model.decoder.embed_tokens.weight": W["dec.tok_emb"],
          "model.decoder.embed_positions.weight": W["dec.pos_emb"]}

    def attn(dst, src):
        for a, b in (("q_proj", "q"), ("k_proj", "k"), ("v_proj", "v"), ("out_proj", "o")):
            sd[f"{dst}.{a}.weight"] = W[f"{src}.{b}.w"]
            if b != "k":
                sd[f"{dst}.{a}.bias"] = W[f"{src}.{b}.b"]

    def ln(dst, src):
        sd[dst + ".weight"], sd[dst + ".bias"] = W[src + ".g"], W[src + ".b"]

    def mlp(dst, src):
        for f in ("fc1", "fc2"):
            sd[f"{dst}.{f}.weight"] = W[f"{src}.mlp.{f}.w"]
            sd[f"{dst}.{f}.bias"] = W[f"{src}.mlp.{f}.b"]

    for i in range(shape.n_enc):
        p, q = f"model.encoder.layers.{i}", f"enc.{i}"
        ln(p + ".self_attn_layer_norm", q + ".attn_ln")
        attn(p + ".self_attn", q + ".attn")
        ln(p + ".final_layer_norm", q + ".mlp_ln")
        mlp(p, q)
    ln("model.encoder.layer_norm", "enc.ln_post")
    for i in range(shape.n_dec):
        p, q = f"model.decoder.layers.{i}", f"dec.{i}"
        ln(p + ".self_attn_layer_norm", q + ".attn_ln")
        attn(p + ".self_attn", q + ".attn")
        ln(p + ".encoder_attn_layer_norm", q + ".cross_ln")
        attn(p + ".encoder_attn", q + ".cross")
        ln(p + ".final_layer_norm", q + ".mlp_ln")
        mlp(p, q)
    ln("model.decoder.layer_norm", "dec.ln")
    sd = {k: torch.from_numpy(np.asarray(v, np.float64)) for k, v in sd.items()}
    missing, unexpected = m.load_state_dict(sd, strict=False)
    assert not unexpected
    assert set(missing) <= {"model.encoder.embed_positions.weight", "proj_out.weight"}
    # the library's own sinusoid table, built in float64
    prev = torch.get_default_dtype()
    torch.set_default_dtype(torch.float64)
    try:
        pe = tfm.sinusoids(1500, shape.d)
    finally:
        torch.set_default_dtype(prev)
    with torch.no_grad():
        m.model.encoder.embed_positions.weight.copy_(pe)
    assert m.proj_out.weight.data_ptr() == m.model.decoder.embed_tokens.weight.data_ptr()  # tied head
    return m


def test_network_matches_library_whisper(weights, segments):
    m = _hf_model(SMALL_SHAPE, weights)
    feats = np.stack([oracle.log_mel_segment(s.audio, 80) for s in segments])
    E = M.encoder(weights, SMALL_SHAPE, feats)
    with torch.no_grad():
        lib_e = m.model.encoder(torch.from_numpy(feats)).last_hidden_state.numpy()
    assert np.abs(E - lib_e).max() <= 1e-12 * np.abs(E).max()
    ckv = M.cross_kv(weights, SMALL_SHAPE, E)
    for b in range(len(segments)):
        toks, lg = M.greedy(weights, SMALL_SHAPE, M._seg_ckv(ckv, b), PROMPT, 6)
        ids = torch.tensor([PROMPT + [int(t) for t in toks[:-1]]])
        with torch.no_grad():
            lib = m(input_features=torch.from_numpy(feats[b:b + 1]),
                    decoder_input_ids=ids).logits[0].numpy()
        assert np.abs(lib[len(PROMPT) - 1:] - lg).max() <= 1e-10 * np.abs(lg).max()


# ------------------------------------------------------- decoding invariants

def test_cached_decode_equals_full_recompute(weights, segments):
    feats = np.stack([oracle.log_mel_segment(segments[0].audio, 80)])
    ckv = M._seg_ckv(M.cross_kv(weights, SMALL_SHAPE, M.encoder(weights, SMALL_SHAPE, feats)), 0)
    t1, l1 = M.greedy(weights, SMALL_SHAPE, ckv, PROMPT, 6, cached=True)
    t2, l2 = M.greedy(weights, SMALL_SHAPE, ckv, PROMPT, 6, cached=False)
    assert np.array_equal(t1, t2)
    assert np.abs(l1 - l2).max() <= 1e-12 * np.abs(l2).max()
    forced = [7, 8, 9, 10, 11, 12]
    t3, l3 = M.greedy(weights, SMALL_SHAPE, ckv, PROMPT, 6, forced=forced, cached=True)
    t4, l4 = M.greedy(weights, SMALL_SHAPE, ckv, PROMPT, 6, forced=forced, cached=False)
    assert np.array_equal(t3, t4) and np.abs(l3 - l4).max() <= 1e-12 * np.abs(l4).max()
    assert np.array_equal(l3[0], l1[0])       # forcing only changes what comes after token 1
    # teacher forcing with the model's own tokens reproduces the free run
    t5, l5 = M.greedy(weights, SMALL_SHAPE, ckv, PROMPT, 6, forced=t1, cached=True)
    assert np.array_equal(t5, t1) and np.array_equal(l5, l1)


def test_batch_equals_solo(weights, segments):
    batch = M.transcribe(weights, SMALL_SHAPE, segments, return_logits=True)
    for s, r in zip(segments, batch):
        solo = M.transcribe(weights, SMALL_SHAPE, [s], return_logits=True)[0]
        assert r["segment_id"] == s.segment_id and r["user_id"] == s.user_id
        assert np.array_equal(r["tokens"], solo["tokens"])
        assert np.abs(r["logits"] - solo["logits"]).max() <= 1e-12 * np.abs(solo["logits"]).max()


def test_greedy_ties_take_lowest_id(weights, segments):
    feats = np.stack([oracle.log_mel_segment(segments[0].audio, 80)])
    ckv = M._seg_ckv(M.cross_kv(weights, SMALL_SHAPE, M.encoder(weights, SMALL_SHAPE, feats)), 0)
    # rows 500 and 600 are never fed, so they only act as output directions;
    # make both the same large multiple of the final hidden state
    cache = M.DecoderCache(SMALL_SHAPE)
    for t in PROMPT[:-1]:
        M.decoder_step(weights, SMALL_SHAPE, t, cache, ckv)
    W2 = dict(weights.values)
    lg = M.decoder_step(weights, SMALL_SHAPE, PROMPT[-1], cache, ckv)
    emb = np.asarray(W2["dec.tok_emb"], np.float64)
    # recover z from the logits with a least-squares solve against the embedding
    z = np.linalg.lstsq(emb, lg, rcond=None)[0]
    emb = emb.copy()
    emb[600] = emb[500] = 50.0 * z / (z @ z)
    W2["dec.tok_emb"] = emb
    toks, lg2 = M.greedy(W2, SMALL_SHAPE, ckv, PROMPT, 1)
    assert lg2[0, 500] == lg2[0, 600] and lg2[0, 500] == lg2[0].max()
    assert toks[0] == 500


def test_transcribe_batch_maps_ids_in_input_order(weights):
    segs = synth.poisson_users(SMALL_SHAPE, 3, 5, 5.0, 2, 4, seed=3)
    for s in segs:
        s.prompt = list(PROMPT)
    res = M.transcribe_batch(weights, SMALL_SHAPE, segs, max_batch=2)
    assert [(r["user_id"], r["segment_id"]) for r in res] == [(s.user_id, s.segment_id) for s in segs]
    assert [len(r["tokens"]) for r in res] == [s.max_new_tokens for s in segs]
    solo = [M.transcribe(weights, SMALL_SHAPE, [s])[0]["tokens"] for s in segs]
    assert all(np.array_equal(a["tokens"], b) for a, b in zip(res, solo))


def test_prompt_length_validation(weights):
    with pytest.raises(ValueError):
        M.greedy(weights, SMALL_SHAPE, None, [], 3)
    with pytest.raises(ValueError):
        M.greedy(weights, SMALL_SHAPE, None, PROMPT, 445)


# ---------------------------------------------------------------- logit filters and end of text

def test_pick_token_is_the_filtered_argmax():
    """By definition: the choice is allowed, no allowed id has a larger
    logit, and no allowed id with an equal logit is smaller (small integer
    logits make ties common)."""
    g = _rng(11)
    for trial in range(200):
        lg = g.integers(-3, 4, 40).astype(np.float64)
        sup = set(g.choice(40, g.integers(0, 10), replace=False).tolist())
        beg = set(g.choice(40, g.integers(0, 10), replace=False).tolist())
        step = int(g.integers(0, 3))
        banned = sup | (beg if step == 0 else set())
        if len(banned) == 40:
            continue
        t = M.pick_token(lg, step, sup, beg)
        assert t not in banned
        allowed = [i for i in range(40) if i not in banned]
        assert lg[t] == max(lg[i] for i in allowed)
        assert t == min(i for i in allowed if lg[i] == lg[t])


def _ref_run(weights, segments, n=6):
    s = segments[0]
    E = M.encoder(weights, SMALL_SHAPE, oracle.log_mel_segment(s.audio, SMALL_SHAPE.n_mels)[None])
    ckv = M._seg_ckv(M.cross_kv(weights, SMALL_SHAPE, E), 0)
    toks, lg = M.greedy(weights, SMALL_SHAPE, ckv, s.prompt, n)
    return ckv, s.prompt, toks, lg


def test_end_of_text_truncates_the_unconstrained_run(weights, segments):
    ckv, prompt, toks, lg = _ref_run(weights, segments)
    # the first position holding a token not seen before it (position 0 if none later)
    k = next((i for i in range(1, len(toks)) if toks[i] not in toks[:i]), 0)
    got, glg = M.greedy(weights, SMALL_SHAPE, ckv, prompt, len(toks), eot=int(toks[k]))
    assert np.array_equal(got, toks[:k])
    assert len(glg) == k + 1 and np.array_equal(glg, lg[:k + 1])   # one row per choice, the stop included


def test_suppressing_the_choice_takes_the_runner_up(weights, segments):
    ckv, prompt, toks, lg = _ref_run(weights, segments)
    got, glg = M.greedy(weights, SMALL_SHAPE, ckv, prompt, 1, suppress={int(toks[0])})
    order = np.argsort(-lg[0], kind="stable")
    assert order[0] == toks[0] and got[0] == order[1]
    got_b, _ = M.greedy(weights, SMALL_SHAPE, ckv, prompt, 1, suppress_begin={int(toks[0])})
    assert got_b[0] == order[1]


def test_begin_suppression_applies_to_the_first_choice_only(weights, segments):
    """With the first choice begin-suppressed, the run takes the runner-up r
    first and then continues exactly as the unfiltered run whose prompt ends
    with r (the begin list no longer applies)."""
    ckv, prompt, toks, lg = _ref_run(weights, segments)
    r = int(np.argsort(-lg[0], kind="stable")[1])
    got, _ = M.greedy(weights, SMALL_SHAPE, ckv, prompt, len(toks), suppress_begin={int(toks[0])})
    rest, _ = M.greedy(weights, SMALL_SHAPE, ckv, list(prompt) + [r], len(toks) - 1)
    assert got[0] == r and np.array_equal(got[1:], rest)
