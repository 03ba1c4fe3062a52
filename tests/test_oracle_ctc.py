"""Pins of the CTC oracle (oracle/ctc.py) to the definitions it follows.

* collapse is the CTC many-to-one map: checked on hand-worked paths, and as
  the inverse of path generation (any label sequence, expanded into a valid
  frame path by repeating labels and inserting blanks, collapses back to
  itself);
* best_path is best-path decoding: on tiny cases, brute force over every
  frame path finds no path more probable than the per-frame argmax, and ties
  go to the lowest id;
* valid_frames counts the 320-sample encoder frames that cover the audio;
* ctc_logits is affine in the encoder output.
"""
import itertools

import numpy as np
import pytest

from oracle import ctc


@pytest.mark.parametrize("path,labels", [
    ([], []),
    ([0, 0, 0], []),
    ([3], [3]),
    ([1, 1, 0, 1], [1, 1]),            # a blank separates two equal labels
    ([1, 1, 1, 1], [1]),                # a run merges
    ([2, 3, 3, 0, 0, 3, 4], [2, 3, 3, 4]),
    ([0, 5, 0, 5, 5, 0], [5, 5]),
    ([7, 8, 9], [7, 8, 9]),
])
def test_collapse_hand_worked(path, labels):
    assert ctc.collapse(path) == labels


def _expand(labels, rng, max_rep=3, p_blank=0.4):
    """A random valid CTC path for `labels`: each label repeated 1..max_rep
    times, blanks inserted at random, and always one blank between equal
    neighbours."""
    path = []
    for k, y in enumerate(labels):
        if rng.random() < p_blank or (k > 0 and labels[k - 1] == y):
            path += [0] * int(rng.integers(1, 3))
        path += [y] * int(rng.integers(1, max_rep + 1))
    if rng.random() < p_blank:
        path += [0] * int(rng.integers(1, 3))
    return path


def test_collapse_inverts_path_generation():
    rng = np.random.default_rng(7)
    for _ in range(500):
        n = int(rng.integers(0, 12))
        labels = [int(v) for v in rng.integers(1, 5, n)]   # small alphabet: many equal neighbours
        assert ctc.collapse(_expand(labels, rng)) == labels


def test_best_path_is_most_probable_path_by_brute_force():
    rng = np.random.default_rng(3)
    for _ in range(30):
        T, V = int(rng.integers(1, 5)), int(rng.integers(2, 4))
        logits = rng.normal(size=(T, V))
        logp = logits - np.log(np.exp(logits).sum(axis=1, keepdims=True))
        best = max(itertools.product(range(V), repeat=T), key=lambda p: sum(logp[t, p[t]] for t in range(T)))
        assert ctc.best_path(logits, T) == list(best)


def test_best_path_ties_go_to_lowest_id_and_respects_frame_count():
    lg = np.array([[1.0, 2.0, 2.0], [0.5, 0.5, 0.1], [3.0, 0.0, 3.0]])
    assert ctc.best_path(lg, 3) == [1, 0, 0]
    assert ctc.best_path(lg, 2) == [1, 0]
    assert ctc.best_path(lg, 0) == []


@pytest.mark.parametrize("n,frames", [(1, 1), (320, 1), (321, 2), (640, 2), (16000, 50), (479999, 1500),
                                      (480000, 1500)])
def test_valid_frames(n, frames):
    assert ctc.valid_frames(n) == frames


def test_ctc_logits_affine_in_encoder_output():
    rng = np.random.default_rng(5)
    d, V = 12, 7
    W = {"ctc.w": rng.normal(size=(V, d)), "ctc.b": rng.normal(size=V)}
    E1, E2 = rng.normal(size=(4, d)), rng.normal(size=(4, d))
    a, b = 0.3, -1.7
    lhs = ctc.ctc_logits(W, a * E1 + b * E2) - W["ctc.b"]
    rhs = a * (ctc.ctc_logits(W, E1) - W["ctc.b"]) + b * (ctc.ctc_logits(W, E2) - W["ctc.b"])
    assert np.allclose(lhs, rhs, rtol=1e-12, atol=1e-12)
    # a head that copies the first V features of the frame returns them plus the bias
    W2 = {"ctc.w": np.eye(V, d), "ctc.b": W["ctc.b"]}
    assert np.allclose(ctc.ctc_logits(W2, E1), E1[:, :V] + W["ctc.b"])


def _label_probs_brute_force(logits):
    """P(y) for every label sequence y: the sum over all frame paths that
    collapse to y of the product of per-frame softmax probabilities."""
    T, V = logits.shape
    p = np.exp(logits - logits.max(axis=1, keepdims=True))
    p /= p.sum(axis=1, keepdims=True)
    out = {}
    for path in itertools.product(range(V), repeat=T):
        y = tuple(ctc.collapse(path))
        out[y] = out.get(y, 0.0) + float(np.prod([p[t, path[t]] for t in range(T)]))
    return out


def test_prefix_beam_search_unpruned_is_exact_by_brute_force():
    """With every label a candidate at every frame and a beam wider than the
    number of prefixes, prefix beam search returns the most probable label
    sequence (brute force over all frame paths)."""
    rng = np.random.default_rng(11)
    for _ in range(25):
        T, V = int(rng.integers(1, 5)), int(rng.integers(2, 4))
        logits = rng.normal(size=(T, V)) * 2
        probs = _label_probs_brute_force(logits)
        best = max(probs, key=probs.get)
        labels, _ = ctc.prefix_beam_search(logits, T, beam=10_000, per_frame=V - 1)
        assert tuple(labels) == best


def _restricted_label_probs(logits, per_frame):
    """P(y) over the candidate-restricted lattice: frame t may emit only the
    blank or one of its per_frame most probable non-blank labels (lowest id
    on ties); every path through those choices that collapses to y adds the
    product of its per-frame softmax probabilities (brute force)."""
    T, V = logits.shape
    p = np.exp(logits - logits.max(axis=1, keepdims=True))
    p /= p.sum(axis=1, keepdims=True)
    allowed = [[0] + sorted(range(1, V), key=lambda c: (-p[t, c], c))[:per_frame] for t in range(T)]
    out = {}
    for path in itertools.product(*allowed):
        y = tuple(ctc.collapse(path))
        out[y] = out.get(y, 0.0) + float(np.prod([p[t, path[t]] for t in range(T)]))
    return out


def test_prefix_beam_search_pruned_candidates_by_brute_force():
    """With fewer candidates than labels per frame (per_frame < V - 1) and a
    beam wider than the number of prefixes, the search returns the most
    probable label sequence of the candidate-restricted lattice."""
    rng = np.random.default_rng(14)
    for _ in range(25):
        T, V = int(rng.integers(1, 5)), int(rng.integers(4, 6))
        per_frame = int(rng.integers(1, V - 2))
        logits = rng.normal(size=(T, V)) * 2
        probs = _restricted_label_probs(logits, per_frame)
        best = max(probs, key=probs.get)
        labels, _ = ctc.prefix_beam_search(logits, T, beam=10_000, per_frame=per_frame)
        assert tuple(labels) == best


def test_prefix_beam_search_tie_order_hand_worked():
    """Two frames, blank and labels 1, 2, all logits equal (every id has
    probability 1/3), beam 2, both labels candidates. Frame 0 yields (), (1)
    and (2) at 1/3 each; the tie order (stays, then extensions in candidate
    order) keeps () and (1). Frame 1 then gives (1) = 1/9 (blank after it) +
    1/9 (its label repeated) + 1/9 (label 1 after the empty prefix) = 1/3,
    and (), (2), (1, 2) 1/9 each: the output is [1], and the smallest margin
    is 0 (the tie at frame 0). Keeping (2) instead would give [2]."""
    labels, margin = ctc.prefix_beam_search(np.zeros((2, 3)), 2, beam=2, per_frame=2)
    assert labels == [1] and margin == 0.0
    # with a beam of one the empty prefix (the first stay) wins every tie
    assert ctc.prefix_beam_search(np.zeros((2, 3)), 2, beam=1, per_frame=2) == ([], 0.0)


def test_prefix_beam_search_pruned_properties():
    """A pruned search returns a valid label sequence, its margin is
    non-negative, and widening the beam never lowers the returned
    sequence's exact probability on these cases."""
    rng = np.random.default_rng(13)
    for _ in range(20):
        T, V = 4, 4
        logits = rng.normal(size=(T, V)) * 2
        probs = _label_probs_brute_force(logits)
        l1, m1 = ctc.prefix_beam_search(logits, T, beam=1, per_frame=1)
        l3, m3 = ctc.prefix_beam_search(logits, T, beam=8, per_frame=3)
        assert all(1 <= c < V for c in l1 + l3) and m1 >= 0 and m3 >= 0
        assert probs[tuple(l3)] >= probs[tuple(l1)] - 1e-12
    assert ctc.prefix_beam_search(np.zeros((0, 3)), 0, 4, 2) == ([], float("inf"))
