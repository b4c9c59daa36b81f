"""Seeded synthetic router inputs: prompts of five task families and random router weights.

The paper routes prompts of five task families (reasoning, generation, retrieval, code,
translation); the suites themselves are not used. Prompts here are built from templates of this
module with pseudo-words drawn from random syllables, so that each family carries the surface
structure the router's descriptors look at (digits and operators, option labels, numbered lists,
code fences and punctuation, wh-questions, a translation request) at a spread of lengths, up to
the paper's 2,048-token prompt (about 8 KiB of text).

Draws use numpy's ``default_rng`` keyed by a list:
* prompt i of a set: ``[seed, i]``; family i % 5 unless given;
* router weights: ``[seed, m]`` for m = 0..6 (projection, W1, b1, W2, b2, W3, b3);
* proxy-LM mean log-probabilities: ``[seed, 7]``, uniform in [-4, -1].
"""
from __future__ import annotations

import numpy as np

__all__ = ["FAMILIES", "prompt", "prompts", "pack", "router_weights", "proxy_logprobs",
           "ROUTER_SHAPE"]

FAMILIES = ("reasoning", "generation", "retrieval", "code", "translation")
ROUTER_SHAPE = {"n_bins": 2048, "proj_dim": 256, "hidden1": 512, "hidden2": 256, "n_tasks": 5}

_ONSETS = ["b", "c", "d", "f", "g", "h", "k", "l", "m", "n", "p", "r", "s", "t", "v", "w", "z",
           "br", "st", "tr", "ch", "sh", "pl"]
_VOWELS = ["a", "e", "i", "o", "u", "ai", "ou", "ea"]
_LANGS = ["German", "French", "Spanish", "Italian"]


def _word(rng, cap=False):
    w = "".join(rng.choice(_ONSETS) + rng.choice(_VOWELS) for _ in range(int(rng.integers(1, 4))))
    return w.capitalize() if cap else w


def _sentence(rng, n=None):
    n = int(rng.integers(4, 14)) if n is None else n
    words = [_word(rng) for _ in range(n)]
    words[0] = words[0].capitalize()
    return " ".join(words) + "."


def _para(rng, n_sent):
    return " ".join(_sentence(rng) for _ in range(n_sent))


def _reasoning(rng, n_sent):
    a, b, c = (int(v) for v in rng.integers(2, 999, 3))
    op = rng.choice(["+", "-", "*", "/"])
    body = _para(rng, n_sent) + f" If {_word(rng)} has {a} {_word(rng)}s and gets {b} {op} {c} more,"
    body += f" how many {_word(rng)}s are there?"
    if rng.random() < 0.5:
        opts = [int(v) for v in rng.integers(1, 5000, 4)]
        style = rng.integers(0, 3)
        lab = [("A.", "B.", "C.", "D."), ("A)", "B)", "C)", "D)"), ("(A)", "(B)", "(C)", "(D)")][style]
        body += "\n" + "\n".join(f"{lab[k]} {opts[k]}" for k in range(4)) + "\nAnswer:"
    else:
        body += f" Show the steps: {a} {op} {b} = ?"
    return body


def _generation(rng, n_sent):
    body = f"Write a {_word(rng)} about {_word(rng)} and {_word(rng)}. " + _para(rng, n_sent)
    if rng.random() < 0.5:
        body += "\nCover these points:\n" + "\n".join(
            f"{k + 1}. {_sentence(rng, int(rng.integers(3, 8)))}" for k in range(int(rng.integers(2, 6))))
    return body


def _retrieval(rng, n_sent):
    wh = rng.choice(["Who", "When", "Where", "Which"])
    q = f"{wh} {_word(rng)} the {_word(rng)} of {_word(rng, True)} {_word(rng, True)}?"
    ctx = _para(rng, max(0, n_sent - 1))
    return (ctx + "\n" + q) if ctx else q


def _code(rng, n_sent):
    name = "_".join(_word(rng) for _ in range(2))
    args = ", ".join(_word(rng) for _ in range(int(rng.integers(1, 4))))
    doc = _sentence(rng)
    lines = [f"def {name}({args}):", f'    """{doc}"""']
    for _ in range(int(rng.integers(1, 2 + n_sent))):
        v = _word(rng)
        lines.append(f"    {v} = [{_word(rng)}[i] * {int(rng.integers(1, 99))} for i in range(len({_word(rng)}))]")
        lines.append(f"    if {v} and {v}[0] >= {int(rng.integers(0, 9))}: {{'{_word(rng)}': {v}}}")
    lines.append(f"    return {_word(rng)}")
    fence = rng.random() < 0.6
    text = "Complete the function. " + _sentence(rng) + "\n"
    text += ("```python\n" if fence else "") + "\n".join(lines) + ("\n```" if fence else "")
    return text


def _translation(rng, n_sent):
    lang = rng.choice(_LANGS)
    verb = rng.choice(["Translate", "translate", "Translation of"])
    return f"{verb} the following text into {lang}: " + _para(rng, n_sent)


_MAKERS = (_reasoning, _generation, _retrieval, _code, _translation)


def prompt(seed: int, i: int, family: int | None = None, n_sent: int | None = None) -> bytes:
    """Prompt i of the set keyed by seed, as UTF-8 bytes."""
    rng = np.random.default_rng([seed, i])
    fam = i % len(FAMILIES) if family is None else family
    if n_sent is None:
        # lengths from a few words to a few KiB (log-uniform sentence count)
        n_sent = int(np.exp(rng.uniform(0.0, np.log(60.0))))
    return _MAKERS[fam](rng, n_sent).encode("utf-8")


def prompts(n: int, seed: int = 11, family: int | None = None, n_sent: int | None = None):
    return [prompt(seed, i, family, n_sent) for i in range(n)]


def pack(texts):
    """Concatenated bytes (uint8) and int32 offsets [n + 1]."""
    offs = np.zeros(len(texts) + 1, np.int32)
    for i, t in enumerate(texts):
        offs[i + 1] = offs[i] + len(t)
    buf = np.frombuffer(b"".join(texts), np.uint8).copy() if texts else np.zeros(0, np.uint8)
    return buf, offs


def router_weights(seed: int = 12, n_bins: int = 2048, proj_dim: int = 256, hidden1: int = 512,
                   hidden2: int = 256, n_tasks: int = 5) -> dict:
    """Random router weights (float32, row-major [out][in]): a frozen N(0, 16) projection
    [proj_dim][n_bins], He-scaled hidden layers, biases 0.01 N(0, 1)."""
    f = proj_dim + 11

    def g(m, shape, std):
        return (np.random.default_rng([seed, m]).standard_normal(shape) * std).astype(np.float32)

    return {"proj": g(0, (proj_dim, n_bins), 4.0),
            "w1": g(1, (hidden1, f), np.sqrt(2.0 / f)), "b1": g(2, (hidden1,), 0.01),
            "w2": g(3, (hidden2, hidden1), np.sqrt(2.0 / hidden1)), "b2": g(4, (hidden2,), 0.01),
            "w3": g(5, (n_tasks, hidden2), np.sqrt(1.0 / hidden2)), "b3": g(6, (n_tasks,), 0.01)}


def proxy_logprobs(n: int, seed: int = 12) -> np.ndarray:
    return np.random.default_rng([seed, 7]).uniform(-4.0, -1.0, n).astype(np.float32)
