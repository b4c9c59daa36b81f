"""Seeded random shapes against the oracle: widths, head counts and group sizes, head_dim 64 and
128, FFN widths, raw (unclosed) masks with random keep rates, ragged prompt lengths after random
prior positions, batches 1-8, and LM heads whose vocabularies span several argmax chunks. Each
case is an independent draw from a fixed seed, so a failure names its seed and shape."""
import numpy as np
import pytest
import torch

import synth
from tests.gpu_case import Case, PrefillCase
from tests.helpers import assert_parity
from tests.test_gpu_generate import _compare, _run

pytestmark = pytest.mark.gpu


def _shape(rng, vocab=0):
    dh = int(rng.choice([64, 128]))
    hkv = int(rng.integers(1, 5))
    r = int(rng.choice([1, 2, 4, 8]))
    d = 16 * int(rng.integers(2, 49))
    f = 16 * int(rng.integers(1, 97))
    layers = int(rng.integers(1, 3))
    return synth.tiny_shape(d=d, hq=r * hkv, hkv=hkv, dh=dh, f=f, layers=layers, vocab=vocab)


def _mask(rng, sh, seed):
    p = rng.uniform(0.3, 1.0, size=3)
    return synth.raw_mask(sh, seed, p_q=p[0], p_kv=p[1], p_f=p[2])


@pytest.mark.parametrize("seed", range(48))
def test_random_prefill(seed):
    rng = np.random.default_rng([seed, 11])
    sh = _shape(rng, vocab=int(rng.choice([0, 0, 700])))
    T, pos0 = int(rng.integers(1, 301)), int(rng.integers(0, 201))
    print(f"case random prefill seed={seed} {sh} T={T} pos0={pos0}", flush=True)
    case = PrefillCase(sh, _mask(rng, sh, seed), T, pos0)
    got, want = case.run(), case.oracle()
    assert_parity(got, want, what=f"random prefill seed {seed}")


@pytest.mark.parametrize("seed", range(48))
def test_random_decode(seed):
    rng = np.random.default_rng([seed, 12])
    sh = _shape(rng, vocab=int(rng.choice([0, 0, 700])))
    batch, pos = int(rng.integers(1, 9)), int(rng.integers(0, 400))
    print(f"case random decode seed={seed} {sh} B={batch} pos={pos}", flush=True)
    case = Case(sh, _mask(rng, sh, seed), batch, pos)
    got, want = case.run(), case.oracle()
    assert_parity(got, want, what=f"random decode seed {seed}")


@pytest.mark.parametrize("seed", range(8))
def test_random_request_multichunk_argmax(seed):
    """Requests whose vocabularies (4097 to 9000) span two or three argmax chunks of 4096."""
    rng = np.random.default_rng([seed, 13])
    sh = _shape(rng, vocab=int(rng.integers(4097, 9001)))
    T, n_new = int(rng.integers(1, 65)), int(rng.integers(1, 9))
    print(f"case random request seed={seed} {sh} T={T} n_new={n_new}", flush=True)
    got, gpu_rows, want_rows, last = _run(sh, _mask(rng, sh, seed), T, n_new)
    assert len(got) == n_new + 1
    _compare(got, gpu_rows, want_rows, last)


@pytest.mark.parametrize("seed", range(8))
def test_random_shared_store(seed):
    """Shared-store plans over a groupwise store (widths in multiples of 256, retained channels in
    aligned blocks of 16): a prefill and a batched decode step against the oracle."""
    rng = np.random.default_rng([seed, 14])
    dh = int(rng.choice([64, 128]))
    hkv = int(rng.integers(1, 5))
    r = int(rng.choice([1, 2, 4, 8]))
    while (r * hkv * dh) % 256:
        hkv += 1
    d, f = 256 * int(rng.integers(1, 4)), 256 * int(rng.integers(1, 7))
    sh = synth.tiny_shape(d=d, hq=r * hkv, hkv=hkv, dh=dh, f=f, layers=int(rng.integers(1, 3)))
    p = rng.uniform(0.3, 1.0, size=3)
    mask = synth.raw_mask(sh, seed, p_q=p[0], p_kv=p[1], p_f=p[2], block=16)
    T, pos0 = int(rng.integers(1, 200)), int(rng.integers(0, 100))
    batch, pos = int(rng.integers(1, 9)), int(rng.integers(0, 300))
    print(f"case random shared seed={seed} {sh} T={T} pos0={pos0} B={batch} pos={pos}", flush=True)
    pf = PrefillCase(sh, mask, T, pos0, shared=True)
    assert_parity(pf.run(), pf.oracle(), what=f"random shared prefill seed {seed}")
    dc = Case(sh, mask, batch, pos, shared=True)
    assert_parity(dc.run(), dc.oracle(), what=f"random shared decode seed {seed}")
