"""Oracle for router inference and dense-fallback dispatch (test infrastructure only).

Paper, Sec. "Dependency-Closed Masks and Cache-Consistent Routing" and the appendix paragraph
"Router feature specification": each user turn is routed once. An MLP with two hidden layers
(512 and 256 wide) turns the prompt's feature vector into task logits, which are divided by a
temperature and normalised; a turn whose top probability falls short of tau (0.85) goes to the
dense INT8 plan, any other turn to its top task's plan. That plan then handles the whole turn
(prefill and decode), and cached K/V rows only carry over to a turn served by the same closed
mask. Appendix
"Routing, Calibration, and Task-Switching Robustness", Eq. for L(tau): the mixture-implied decode
latency u L_sparse + (1 - u) L_dense, u the fraction of turns on the sparse path.

The feature vector (appendix paragraph above), in this order:
  (i)   bag of character n-grams hashed into n_bins (2,048) bins, projected to proj_dim (256) by a
        frozen random map R [proj_dim][n_bins];
  (ii)  prompt length and the mean token log-probability of the prompt under a small proxy LM
        (the proxy LM is outside this computation: its value is an input);
  (iii) counts of digits, operators, code punctuation and question marks;
  (iv)  five task descriptors: a numbered list, a code fence, a "translate" cue, a multiple-choice
        pattern and a retrieval cue.

Readings where the paper is silent (each listed in the design notes):
  * n-grams are byte trigrams of the UTF-8 prompt with ASCII A-Z folded to a-z; a trigram's bin
    is its 32-bit FNV-1a hash (offset basis 2166136261, prime 16777619, xor then multiply per
    byte) modulo n_bins; the hashed vector holds term frequencies count / max(1, n - 2);
  * length feature ln(1 + bytes); each count c enters as ln(1 + c);
  * digits 0-9; operators + - * / = < > % ^; code punctuation { } [ ] ( ) ; _ # ` \\ | &;
  * numbered list: a line (text start or after a newline) opening with 1-3 digits, then '.' or
    ')', then a space; code fence: three backticks; translate cue: "translat" (case-folded);
    multiple-choice pattern: lines opening with the option labels A and B, each written "X.",
    "X)" or "(X)" and followed by a space (labels A-D recognised; upper case); retrieval cue: a
    case-folded "who", "when", "where" or "which" at a word start (text start or after a byte
    that is not an ASCII letter or digit) and not followed by a letter;
  * the MLP is ReLU(W1 f + b1), ReLU(W2 h1 + b2), W3 h2 + b3; p = softmax(z / temperature);
    the task is the lowest index of the largest p; the dense plan (-1) when max p < tau.

Plain Python loops for the text scan; float64 numpy for the arithmetic. Nothing here is shared
with the GPU path.
"""
from __future__ import annotations

import math

import numpy as np

N_SCALAR = 11        # length, log-prob, 4 counts, 5 descriptors

FNV_OFFSET = 2166136261
FNV_PRIME = 16777619
OPERATORS = frozenset(b"+-*/=<>%^")
CODE_PUNCT = frozenset(b"{}[]();_#`\\|&")
RETRIEVAL_WORDS = (b"who", b"when", b"where", b"which")


def fnv1a32(data: bytes) -> int:
    """32-bit FNV-1a of a byte string."""
    h = FNV_OFFSET
    for b in data:
        h ^= b
        h = (h * FNV_PRIME) & 0xFFFFFFFF
    return h


def fold(b: int) -> int:
    return b + 32 if 65 <= b <= 90 else b


def _is_alnum(b: int) -> bool:
    return 48 <= b <= 57 or 65 <= b <= 90 or 97 <= b <= 122


def _is_letter(b: int) -> bool:
    return 65 <= b <= 90 or 97 <= b <= 122


def trigram_counts(text: bytes, n_bins: int) -> np.ndarray:
    """Integer count per bin of the prompt's case-folded byte trigrams."""
    c = np.zeros(n_bins, np.int64)
    t = bytes(fold(b) for b in text)
    for p in range(len(t) - 2):
        c[fnv1a32(t[p:p + 3]) % n_bins] += 1
    return c


def char_counts(text: bytes):
    """(digits, operators, code punctuation, question marks)."""
    d = sum(1 for b in text if 48 <= b <= 57)
    o = sum(1 for b in text if b in OPERATORS)
    c = sum(1 for b in text if b in CODE_PUNCT)
    q = text.count(b"?")
    return d, o, c, q


def _line_starts(text: bytes):
    return [p for p in range(len(text)) if p == 0 or text[p - 1] == 10]


def _numbered_at(text: bytes, s: int) -> bool:
    k = 0
    while k < 3 and s + k < len(text) and 48 <= text[s + k] <= 57:
        k += 1
    if k == 0 or s + k + 1 >= len(text):
        return False
    return text[s + k] in b".)" and text[s + k + 1] == 32


def _option_at(text: bytes, s: int):
    """The option label (0 for A .. 3 for D) that opens the line at s, else None."""
    def ch(i):
        return text[i] if i < len(text) else None
    if ch(s) == 40 and ch(s + 1) is not None and 65 <= ch(s + 1) <= 68 and ch(s + 2) == 41 \
            and ch(s + 3) == 32:
        return ch(s + 1) - 65
    if ch(s) is not None and 65 <= ch(s) <= 68 and ch(s + 1) in (46, 41) and ch(s + 2) == 32:
        return ch(s) - 65
    return None


def descriptors(text: bytes):
    """(numbered list, code fence, translate cue, multiple-choice pattern, retrieval cue) as 0/1."""
    starts = _line_starts(text)
    numbered = any(_numbered_at(text, s) for s in starts)
    labels = {_option_at(text, s) for s in starts}
    mc = 0 in labels and 1 in labels
    fence = b"```" in text
    low = bytes(fold(b) for b in text)
    translate = b"translat" in low
    retrieval = False
    for p in range(len(low)):
        if p > 0 and _is_alnum(low[p - 1]):
            continue
        for w in RETRIEVAL_WORDS:
            if low[p:p + len(w)] == w:
                nxt = low[p + len(w)] if p + len(w) < len(low) else None
                if nxt is None or not _is_letter(nxt):
                    retrieval = True
    return tuple(int(v) for v in (numbered, fence, translate, mc, retrieval))


def features(text: bytes, proxy_logprob: float, proj: np.ndarray, n_bins: int) -> np.ndarray:
    """The router's input vector for one prompt: [R tf (proj_dim), scalars (11)], float64."""
    counts = trigram_counts(text, n_bins)
    tf = counts.astype(np.float64) / max(1, len(text) - 2)
    head = np.asarray(proj, np.float64) @ tf
    d, o, c, q = char_counts(text)
    scal = [math.log1p(len(text)), float(proxy_logprob),
            math.log1p(d), math.log1p(o), math.log1p(c), math.log1p(q),
            *[float(v) for v in descriptors(text)]]
    return np.concatenate([head, np.array(scal, np.float64)])


def mlp_logits(f, w1, b1, w2, b2, w3, b3) -> np.ndarray:
    relu = lambda v: np.maximum(v, 0.0)
    h1 = relu(np.asarray(w1, np.float64) @ f + np.asarray(b1, np.float64))
    h2 = relu(np.asarray(w2, np.float64) @ h1 + np.asarray(b2, np.float64))
    return np.asarray(w3, np.float64) @ h2 + np.asarray(b3, np.float64)


def probabilities(z, temperature: float) -> np.ndarray:
    """softmax(z / temperature), shifted by the maximum."""
    u = np.asarray(z, np.float64) / temperature
    e = np.exp(u - u.max())
    return e / e.sum()


def decide(p, tau: float) -> int:
    """Task index of the largest probability (lowest on ties), or -1 (dense plan) below tau."""
    p = np.asarray(p)
    task = int(np.argmax(p))                  # numpy's argmax returns the first maximum
    return task if p[task] >= tau else -1


def route(text: bytes, proxy_logprob: float, w: dict, temperature: float, tau: float):
    """(features, probabilities, choice) for one prompt; w holds proj, w1, b1, w2, b2, w3, b3."""
    n_bins = w["proj"].shape[1]
    f = features(text, proxy_logprob, w["proj"], n_bins)
    p = probabilities(mlp_logits(f, w["w1"], w["b1"], w["w2"], w["b2"], w["w3"], w["b3"]),
                      temperature)
    return f, p, decide(p, tau)


def mixture_latency(u: float, l_sparse: float, l_dense: float) -> float:
    """Mixture-implied per-token latency at sparse-path usage u."""
    return u * l_sparse + (1.0 - u) * l_dense


def sparse_usage(choices) -> float:
    c = list(choices)
    return sum(1 for v in c if v >= 0) / len(c) if c else 0.0
