"""Pins for the oracle's request loop (prefill, greedy token, decode steps under one plan)."""
import numpy as np

import synth
from oracle import reference as ref

SH = synth.tiny_shape(d=32, hq=4, hkv=2, dh=8, f=48, layers=2, vocab=50, theta=10000.0)


def _setup(mask_seed=None):
    layers = [synth.layer_weights(SH, l) for l in range(SH.n_layers)]
    m = synth.raw_mask(SH, mask_seed) if mask_seed is not None else synth.all_kept_mask(SH)
    closed = ref.close_mask(*m, SH.group_size)
    table, scales = synth.embedding(SH)
    return layers, closed, table, scales


def _caches(S):
    return [(np.zeros((SH.n_kv_heads, S, SH.head_dim)), np.zeros((SH.n_kv_heads, S, SH.head_dim)))
            for _ in range(SH.n_layers)]


def test_greedy_token_takes_the_lowest_of_equal_maxima():
    assert ref.greedy_token(np.array([1.0, 3.0, 3.0, 2.0])) == 1
    assert ref.greedy_token(np.array([-5.0, -1.0, -1.0])) == 1


def test_embedding_is_the_dequantised_row():
    table, scales = synth.embedding(SH)
    ids = [3, 0, 49, 3]
    got = ref.embed_rows(table, scales, ids)
    assert got.shape == (4, SH.d_model)
    assert np.array_equal(got[0], got[3])
    assert np.allclose(got[1], table[0].astype(np.float64) * float(scales[0]), rtol=0, atol=0)
    # per-row quantisation keeps every row within half a step of its N(0, 1) source
    src = np.random.default_rng([0, SH.n_layers, 2]).standard_normal((SH.vocab, SH.d_model), dtype=np.float32)
    assert np.all(np.abs(ref.embed_rows(table, scales, range(SH.vocab)) - src) <= scales[:, None] / 2 + 1e-7)


def test_loop_equals_one_prefill_of_the_whole_sequence():
    """The greedy ids of the loop are the argmaxes of a single prefill over prompt + generated
    tokens at positions T-1 .. T-1+n (position bookkeeping and token feeding)."""
    for mask_seed in (None, 3):
        layers, closed, table, scales = _setup(mask_seed)
        prompt = synth.prompt_ids(7, SH.vocab)
        n = 5
        toks, rows = ref.generate(lambda l: layers[l], closed, table, scales, prompt, n, _caches(16),
                                  SH, synth.final_norm(SH), synth.lm_head(SH))
        assert len(toks) == n + 1
        seq = np.concatenate([prompt, toks[:-1]])
        full = ref.prefill_stack(lambda l: layers[l], closed, ref.embed_rows(table, scales, seq),
                                 _caches(16), 0, SH, synth.final_norm(SH), synth.lm_head(SH))
        assert np.array_equal(full[len(prompt) - 1:].argmax(axis=1), toks)
        assert np.allclose(full[len(prompt) - 1:], rows, rtol=1e-10, atol=1e-10)


def test_no_decode_steps_gives_the_prefill_token():
    layers, closed, table, scales = _setup()
    prompt = synth.prompt_ids(4, SH.vocab, seed=9)
    toks, rows = ref.generate(lambda l: layers[l], closed, table, scales, prompt, 0, _caches(8), SH,
                              synth.final_norm(SH), synth.lm_head(SH))
    full = ref.prefill_stack(lambda l: layers[l], closed, ref.embed_rows(table, scales, prompt),
                             _caches(8), 0, SH, synth.final_norm(SH), synth.lm_head(SH))
    assert toks.tolist() == [int(full[-1].argmax())]
