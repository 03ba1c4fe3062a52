"""Oracle network: conv stem, transformer encoder, greedy decoder with
self- and cross-attention caches, in float64.

TEST INFRASTRUCTURE ONLY (see oracle/__init__.py).

The paper batches independent segments through one encode call and one
generate call with the prompt plus no-timestamps token per segment
(Section 2.3, Listing 1); it does not define the network. The network here
is the public Whisper encoder-decoder:

* stem: conv1d(k3, s1, p1) + GELU, conv1d(k3, s2, p1) + GELU, plus fixed
  sinusoidal positions (timescale increment ln(10000) / (d/2 - 1));
* encoder block: x += MHA(LN x), x += W2 GELU(W1 LN x + b1) + b2, no mask;
  keys carry no bias; a final layer norm;
* decoder block: causal self-attention, cross-attention over the encoder
  output, MLP, all pre-LN; token + learned position embeddings in; final
  layer norm and the transposed token embedding as output head;
* GELU is the erf form; layer norm uses the biased variance and eps 1e-5.

Greedy decoding feeds the prompt, takes the argmax at the prompt's last
position as the first new token, feeds each new token back, and stops after
exactly max_new_tokens tokens (end-of-text is not special). Ties go to the
lowest token id. Weights are read as given and computed in float64;
activations are never rounded.
"""
import math

import numpy as np
from scipy.special import erf

from .frontend import log_mel_segment

LN_EPS = 1e-5


def _w(W, name):
    return np.asarray(W[name], dtype=np.float64)


def layer_norm(x, g, b, eps=LN_EPS):
    """(x - mean) / sqrt(var + eps) * g + b over the last axis (biased var)."""
    mu = x.mean(axis=-1, keepdims=True)
    var = ((x - mu) ** 2).mean(axis=-1, keepdims=True)
    return (x - mu) / np.sqrt(var + eps) * g + b


def gelu(x):
    """x * Phi(x) with the exact normal CDF (erf form)."""
    return 0.5 * x * (1.0 + erf(x / math.sqrt(2.0)))


def softmax(s, axis=-1):
    e = np.exp(s - s.max(axis=axis, keepdims=True))
    return e / e.sum(axis=axis, keepdims=True)


def _ln(W, prefix, x):
    return layer_norm(x, _w(W, prefix + ".g"), _w(W, prefix + ".b"))


def _linear(W, prefix, x, bias=True):
    y = x @ _w(W, prefix + ".w").T
    if bias:
        y = y + _w(W, prefix + ".b")
    return y


def _heads(x, n_head):
    """[..., T, d] -> [..., h, T, d/h]"""
    *lead, t, d = x.shape
    return np.swapaxes(x.reshape(*lead, t, n_head, d // n_head), -3, -2)


def _merge(x):
    """[..., h, T, dh] -> [..., T, h*dh]"""
    x = np.swapaxes(x, -3, -2)
    return x.reshape(*x.shape[:-2], x.shape[-2] * x.shape[-1])


def attention(q, k, v, causal=False):
    """softmax(q k^T / sqrt(dh)) v per head; with causal, query i (counted
    from the end, aligned to the last key) sees keys j <= i + (Tk - Tq)."""
    s = q @ np.swapaxes(k, -1, -2) / math.sqrt(q.shape[-1])
    if causal:
        tq, tk = s.shape[-2], s.shape[-1]
        allowed = np.arange(tk)[None, :] <= (np.arange(tq)[:, None] + (tk - tq))
        s = np.where(allowed, s, -np.inf)
    return softmax(s) @ v


def mha(W, prefix, xq, xkv, n_head, causal=False):
    """Projections q = xq Wq^T + bq, k = xkv Wk^T (no bias),
    v = xkv Wv^T + bv; per-head attention; output projection with bias."""
    q = _heads(_linear(W, prefix + ".q", xq), n_head)
    k = _heads(_linear(W, prefix + ".k", xkv, bias=False), n_head)
    v = _heads(_linear(W, prefix + ".v", xkv), n_head)
    return _linear(W, prefix + ".o", _merge(attention(q, k, v, causal)))


def _conv1d(x, w, b, stride):
    """x [B, Cin, T], w [Cout, Cin, 3], zero padding 1 each side: output t
    reads inputs stride*t - 1, stride*t, stride*t + 1."""
    t_in = x.shape[-1]
    t_out = (t_in + 2 - 3) // stride + 1
    xp = np.pad(x, ((0, 0), (0, 0), (1, 1)))
    out = np.zeros((x.shape[0], w.shape[0], t_out)) + b[None, :, None]
    for tap in range(3):
        cols = xp[:, :, tap: tap + stride * (t_out - 1) + 1: stride]   # [B, Cin, t_out]
        out += np.einsum("oc,bct->bot", w[:, :, tap], cols)
    return out


def conv_stem(W, mel):
    """[B, n_mels, 3000] -> [B, 1500, d]"""
    h = gelu(_conv1d(mel, _w(W, "enc.conv1.w"), _w(W, "enc.conv1.b"), 1))
    h = gelu(_conv1d(h, _w(W, "enc.conv2.w"), _w(W, "enc.conv2.b"), 2))
    return np.swapaxes(h, 1, 2)


def sinusoid_pe(length, d, max_timescale=10000.0):
    """PE[t, j] = sin(t * r_j), PE[t, d/2 + j] = cos(t * r_j) with
    r_j = exp(-j * ln(max_timescale) / (d/2 - 1)), j < d/2."""
    half = d // 2
    r = np.exp(-np.arange(half) * (math.log(max_timescale) / (half - 1)))
    ang = np.arange(length)[:, None] * r[None, :]
    return np.concatenate([np.sin(ang), np.cos(ang)], axis=1)


def encoder(W, shape, mel):
    """mel [B, n_mels, 3000] -> encoder output E [B, 1500, d]."""
    x = conv_stem(W, np.asarray(mel, dtype=np.float64))
    x = x + sinusoid_pe(x.shape[1], x.shape[2])[None]
    for i in range(shape.n_enc):
        p = f"enc.{i}"
        z = _ln(W, p + ".attn_ln", x)
        x = x + mha(W, p + ".attn", z, z, shape.n_head)
        z = _ln(W, p + ".mlp_ln", x)
        x = x + _linear(W, p + ".mlp.fc2", gelu(_linear(W, p + ".mlp.fc1", z)))
    return _ln(W, "enc.ln_post", x)


def cross_kv(W, shape, E):
    """Per decoder layer: K_c = E Wk^T, V_c = E Wv^T + bv, split into heads:
    a list of (K [B, h, 1500, dh], V [B, h, 1500, dh])."""
    out = []
    for i in range(shape.n_dec):
        p = f"dec.{i}.cross"
        out.append((_heads(_linear(W, p + ".k", E, bias=False), shape.n_head),
                    _heads(_linear(W, p + ".v", E), shape.n_head)))
    return out


def _cross_attend(W, prefix, z, kc, vc, n_head):
    q = _heads(_linear(W, prefix + ".q", z), n_head)
    return _linear(W, prefix + ".o", _merge(attention(q, kc, vc)))


def _mlp(W, p, z):
    return _linear(W, p + ".mlp.fc2", gelu(_linear(W, p + ".mlp.fc1", z)))


def decoder_logits_full(W, shape, tokens, ckv_seg):
    """Full recompute over a token prefix of one segment: logits [P, V] at
    every position 0..P-1. ckv_seg: per layer (K [h, 1500, dh], V [...])."""
    tokens = np.asarray(tokens, dtype=np.int64)
    P = tokens.size
    x = _w(W, "dec.tok_emb")[tokens] + _w(W, "dec.pos_emb")[:P]
    for i in range(shape.n_dec):
        p = f"dec.{i}"
        z = _ln(W, p + ".attn_ln", x)
        x = x + mha(W, p + ".attn", z, z, shape.n_head, causal=True)
        z = _ln(W, p + ".cross_ln", x)
        x = x + _cross_attend(W, p + ".cross", z, ckv_seg[i][0], ckv_seg[i][1], shape.n_head)
        x = x + _mlp(W, p, _ln(W, p + ".mlp_ln", x))
    return _ln(W, "dec.ln", x) @ _w(W, "dec.tok_emb").T


class DecoderCache:
    """Self-attention keys and values of the positions fed so far, per layer
    ([h, t, dh] each)."""

    def __init__(self, shape):
        self.k = [None] * shape.n_dec
        self.v = [None] * shape.n_dec
        self.length = 0


def decoder_step(W, shape, token, cache, ckv_seg):
    """Feed one token at position cache.length; returns logits [V]. The new
    position's self-attention key and value are appended to the cache and
    its query attends to positions 0..cache.length (causal by
    construction)."""
    pos = cache.length
    x = _w(W, "dec.tok_emb")[int(token)] + _w(W, "dec.pos_emb")[pos]
    x = x[None, :]                                                   # [1, d]
    h = shape.n_head
    for i in range(shape.n_dec):
        p = f"dec.{i}"
        z = _ln(W, p + ".attn_ln", x)
        q = _heads(_linear(W, p + ".attn.q", z), h)                   # [h, 1, dh]
        k = _heads(_linear(W, p + ".attn.k", z, bias=False), h)
        v = _heads(_linear(W, p + ".attn.v", z), h)
        cache.k[i] = k if cache.k[i] is None else np.concatenate([cache.k[i], k], axis=1)
        cache.v[i] = v if cache.v[i] is None else np.concatenate([cache.v[i], v], axis=1)
        x = x + _linear(W, p + ".attn.o", _merge(attention(q, cache.k[i], cache.v[i])))
        z = _ln(W, p + ".cross_ln", x)
        x = x + _cross_attend(W, p + ".cross", z, ckv_seg[i][0], ckv_seg[i][1], h)
        x = x + _mlp(W, p, _ln(W, p + ".mlp_ln", x))
    cache.length = pos + 1
    return (_ln(W, "dec.ln", x) @ _w(W, "dec.tok_emb").T)[0]


def pick_token(logits, step, suppress=(), suppress_begin=()):
    """The greedy choice at generated position `step` (0 = first token after
    the prompt) with logit filters: ids in `suppress` can never be chosen,
    ids in `suppress_begin` not at step 0; among the rest, the largest logit,
    lowest id on ties."""
    lg = np.array(logits, dtype=np.float64, copy=True)
    if len(suppress):
        lg[np.asarray(list(suppress), dtype=np.int64)] = -np.inf
    if step == 0 and len(suppress_begin):
        lg[np.asarray(list(suppress_begin), dtype=np.int64)] = -np.inf
    return int(np.argmax(lg))                # first maximum = lowest id on ties


def greedy(W, shape, ckv_seg, prompt, n_new, forced=None, cached=True, eot=None, suppress=(),
           suppress_begin=(), progress=None):
    """Greedy decode of up to n_new tokens after the prompt.

    Token 1 is the choice (pick_token) at the prompt's last position; token
    i+1 the choice after feeding token i (or forced[i-1] when teacher
    forcing). Decoding stops early when the choice is `eot` (end of text,
    not returned). Returns (tokens int64, logits float64): one logits row
    per choice made, i.e. one more row than tokens when stopped by eot.
    progress, if given, is called with the number of choices made so far
    after each one (it takes no part in the computation)."""
    prompt = [int(t) for t in prompt]
    if len(prompt) < 1 or len(prompt) + n_new > shape.n_text_ctx:
        raise ValueError("prompt length + n_new must fit the text context")
    toks, logits = [], []
    if cached:
        cache = DecoderCache(shape)
        for t in prompt[:-1]:
            decoder_step(W, shape, t, cache, ckv_seg)
        nxt = prompt[-1]
        for i in range(n_new):
            lg = decoder_step(W, shape, nxt, cache, ckv_seg)
            g = pick_token(lg, i, suppress, suppress_begin)
            logits.append(lg)
            if progress:
                progress(i + 1)
            if eot is not None and g == eot:
                break
            toks.append(g)
            nxt = g if forced is None else int(forced[i])
    else:
        seq = list(prompt)
        for i in range(n_new):
            lg = decoder_logits_full(W, shape, seq, ckv_seg)[-1]
            g = pick_token(lg, i, suppress, suppress_begin)
            logits.append(lg)
            if eot is not None and g == eot:
                break
            toks.append(g)
            seq.append(g if forced is None else int(forced[i]))
    return np.array(toks, dtype=np.int64), np.stack(logits)


def _seg_ckv(ckv, b):
    return [(k[b], v[b]) for (k, v) in ckv]


def transcribe(W, shape, segments, pad_mode=0, return_logits=False):
    """The batched call of Listing 1: per-segment features on the 30 s
    window, stacked; one encoder pass over the batch; cross-attention keys
    and values; greedy decoding per segment from its own prompt.

    Returns one dict per input segment, in input order:
    {user_id, segment_id, tokens[, logits]}."""
    if len(segments) == 0:
        return []
    feats = np.stack([log_mel_segment(s.audio, shape.n_mels, pad_mode) for s in segments])
    E = encoder(W, shape, feats)
    ckv = cross_kv(W, shape, E)
    out = []
    for b, s in enumerate(segments):
        toks, lg = greedy(W, shape, _seg_ckv(ckv, b), s.prompt, s.max_new_tokens)
        r = {"user_id": s.user_id, "segment_id": s.segment_id, "tokens": toks}
        if return_logits:
            r["logits"] = lg
        out.append(r)
    return out


def transcribe_batch(W, shape, segments, max_batch, pad_mode=0):
    """A queue of segments served in consecutive batches of at most
    max_batch (arrival order), each through `transcribe`; results are mapped
    back to input order."""
    order = sorted(range(len(segments)),
                   key=lambda i: (segments[i].arrival_us, segments[i].user_id,
                                  segments[i].segment_id, i))
    res = [None] * len(segments)
    for s in range(0, len(order), max_batch):
        idx = order[s:s + max_batch]
        for i, r in zip(idx, transcribe(W, shape, [segments[i] for i in idx], pad_mode)):
            res[i] = r
    return res
