"""Pins of the router oracle (features, MLP, temperature softmax, fallback decision, mixture
latency) against values fixed outside it: published FNV-1a test vectors, hand-counted strings,
closed forms of the softmax, and the paper's printed threshold sweep."""
from __future__ import annotations

import json
import math
import os

import numpy as np
import pytest

from oracle import router as R
from synth import text as T

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


# ---- hashing: the FNV-1a reference test vectors


@pytest.mark.parametrize("s,h", [(b"", 0x811C9DC5), (b"a", 0xE40C292C), (b"foobar", 0xBF9CF968)])
def test_fnv1a_published_vectors(s, h):
    assert R.fnv1a32(s) == h


def test_trigram_counts_invariants():
    nb = 2048
    assert R.trigram_counts(b"", nb).sum() == 0
    assert R.trigram_counts(b"ab", nb).sum() == 0
    for s in (b"abc", b"hello world", b"x" * 100):
        assert R.trigram_counts(s, nb).sum() == len(s) - 2
    # one repeated byte: a single bin holds every trigram
    c = R.trigram_counts(b"aaaaaaa", nb)
    assert c.max() == 5 and np.count_nonzero(c) == 1
    # "abcabc" has trigrams abc, bca, cab, abc
    c = R.trigram_counts(b"abcabc", nb)
    assert c[R.fnv1a32(b"abc") % nb] == 2
    assert c[R.fnv1a32(b"bca") % nb] >= 1 and c[R.fnv1a32(b"cab") % nb] >= 1
    # ASCII case folding
    assert np.array_equal(R.trigram_counts(b"Hello WORLD", nb), R.trigram_counts(b"hello world", nb))
    # bytes outside ASCII are hashed as they are
    assert not np.array_equal(R.trigram_counts("äbc".encode(), nb), R.trigram_counts(b"abc", nb))


def test_char_counts_hand_counted():
    s = b"x = 3 + 4*2; f(a)[0] {b} # c ? ?"
    # digits 3 4 2 0; operators = + *; code ; ( ) [ ] { } #; two question marks
    assert R.char_counts(s) == (4, 3, 8, 2)
    assert R.char_counts(b"") == (0, 0, 0, 0)
    assert R.char_counts(b"a/b%c^d<e>f-g") == (0, 6, 0, 0)
    assert R.char_counts(b"`_\\|&") == (0, 0, 5, 0)


D = ("numbered", "fence", "translate", "mc", "retrieval")


@pytest.mark.parametrize("s,flag,val", [
    (b"Steps:\n1. mix\n2. bake", "numbered", 1),
    (b"12) go", "numbered", 1),
    (b"pi is 3.14 here", "numbered", 0),
    (b"1.x", "numbered", 0),
    (b"1234. no", "numbered", 0),
    (b"see\n 1. indented", "numbered", 0),
    (b"```py\nx\n```", "fence", 1),
    (b"`` x ``", "fence", 0),
    (b"Please TRANSLATE this", "translate", 1),
    (b"a translation", "translate", 1),
    (b"transl", "translate", 0),
    (b"Q?\nA. one\nB. two", "mc", 1),
    (b"Q?\n(A) x\n(B) y", "mc", 1),
    (b"A) x\nB) y", "mc", 1),
    (b"A. one only", "mc", 0),
    (b"Q\nA. x\nC. y", "mc", 0),
    (b"a. x\nb. y", "mc", 0),
    (b"A.one\nB.two", "mc", 0),
    (b"Who wrote it", "retrieval", 1),
    (b"where?", "retrieval", 1),
    (b"x-when y", "retrieval", 1),
    (b"ask who", "retrieval", 1),
    (b"WHICH one", "retrieval", 1),
    (b"whom", "retrieval", 0),
    (b"somewhere", "retrieval", 0),
    (b"2who", "retrieval", 0),
    (b"", "retrieval", 0),
])
def test_descriptors_hand_cases(s, flag, val):
    assert R.descriptors(s)[D.index(flag)] == val


def test_features_layout_and_projection():
    nb = 64
    s = b"abcabc? 12 + 3"
    proj = np.zeros((3, nb))
    proj[0, R.fnv1a32(b"abc") % nb] = 1.0       # picks one bin
    proj[1, :] = 1.0                             # sums the term frequencies
    f = R.features(s, -2.5, proj, nb)
    n = len(s)
    assert f.shape == (3 + R.N_SCALAR,)
    assert f[0] == pytest.approx(2 / (n - 2))   # "abc" twice; nothing else in "abcabc? 12 + 3" collides
    assert f[1] == pytest.approx(1.0)
    assert f[2] == 0.0
    assert f[3] == pytest.approx(math.log(1 + n))
    assert f[4] == -2.5
    assert f[5:9] == pytest.approx([math.log(4), math.log(2), 0.0, math.log(2)])
    assert list(f[9:]) == [0, 0, 0, 0, 0]
    # short prompt: no trigrams, projection zero
    g = R.features(b"ab", 0.0, proj, nb)
    assert g[0] == 0.0 and g[1] == 0.0


def test_mlp_hand_network():
    f = np.array([1.0, -2.0])
    w1 = np.array([[1.0, 0.0], [0.0, 1.0], [1.0, 1.0]])
    b1 = np.array([0.0, 0.0, 0.5])
    # h1 = relu([1, -2, -0.5]) = [1, 0, 0]
    w2 = np.array([[2.0, 5.0, 7.0], [-1.0, 0.0, 0.0]])
    b2 = np.array([0.25, 0.0])
    # h2 = relu([2.25, -1]) = [2.25, 0]
    w3 = np.array([[1.0, 3.0], [0.0, 1.0]])
    b3 = np.array([0.0, -1.0])
    assert R.mlp_logits(f, w1, b1, w2, b2, w3, b3) == pytest.approx([2.25, -1.0])


def test_softmax_closed_forms():
    assert R.probabilities(np.zeros(5), 1.0) == pytest.approx([0.2] * 5)
    a = 1.7
    p = R.probabilities([a, 0, 0, 0, 0], 1.0)
    assert p[0] == pytest.approx(math.exp(a) / (math.exp(a) + 4))
    # temperature divides the logits
    z = np.array([0.3, -1.2, 2.0, 0.0, 0.9])
    assert R.probabilities(z, 2.5) == pytest.approx(R.probabilities(z / 2.5, 1.0))
    # large logits do not overflow
    assert R.probabilities([1000.0, 0.0], 1.0) == pytest.approx([1.0, 0.0])
    assert R.probabilities(z, 1e-3).max() == pytest.approx(1.0)


def test_decision_threshold_and_ties():
    tau = 0.85
    a = math.log(tau * 4 / (1 - tau))           # p0 = tau exactly
    assert R.decide(R.probabilities([a + 1e-6, 0, 0, 0, 0], 1.0), tau) == 0
    assert R.decide(R.probabilities([a - 1e-6, 0, 0, 0, 0], 1.0), tau) == -1
    assert R.decide([0.1, 0.45, 0.45], 0.4) == 1
    assert R.decide([0.2] * 5, 0.2) == 0
    assert R.decide([0.2] * 5, 0.21) == -1


def test_route_forced_by_bias():
    w = T.router_weights(seed=3, n_bins=64, proj_dim=8, hidden1=16, hidden2=8)
    w["w3"] = np.zeros_like(w["w3"])
    for task in range(5):
        w["b3"] = np.zeros(5, np.float32)
        w["b3"][task] = 10.0
        for s in T.prompts(5, seed=2):
            assert R.route(s, -1.0, w, 1.0, 0.85)[2] == task
    w["b3"] = np.zeros(5, np.float32)
    f, p, c = R.route(b"anything", -1.0, w, 1.0, 0.85)
    assert c == -1 and p == pytest.approx([0.2] * 5)


def test_mixture_latency_paper_sweep():
    g = json.load(open(os.path.join(GOLDEN, "paper_threshold_sweep.json")))
    half = 0.5 * 10.0 ** -g["printed_decimals"]
    for row in g["rows"]:
        v = R.mixture_latency(row["sparse_use"], g["l_sparse_ms"], g["l_dense_ms"])
        assert abs(v - row["ms_per_token"]) <= half + 1e-9, row
    assert R.mixture_latency(1.0, 3.0, 7.0) == 3.0 and R.mixture_latency(0.0, 3.0, 7.0) == 7.0
    assert R.sparse_usage([0, -1, 3, -1]) == 0.5 and R.sparse_usage([]) == 0.0


def test_synthetic_prompts_carry_family_cues():
    # the generator's structure reaches the descriptors (a check of the inputs, not the oracle)
    fams = {k: T.prompts(40, seed=5, family=k) for k in range(5)}
    frac = lambda k, flag: np.mean([R.descriptors(s)[D.index(flag)] for s in fams[k]])
    assert frac(4, "translate") == 1.0
    assert frac(2, "retrieval") == 1.0
    assert frac(3, "fence") > 0.3
    assert frac(0, "mc") > 0.2
    assert frac(1, "numbered") > 0.2
    assert max(len(s) for k in range(5) for s in fams[k]) > 2000
    buf, offs = T.pack(fams[0])
    assert offs[-1] == len(buf) and bytes(buf[offs[3]:offs[4]]) == fams[0][3]
