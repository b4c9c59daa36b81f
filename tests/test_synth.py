"""Input generators: determinism, the INT8 quantiser's closed-form bounds, BF16 rounding and the
budget mask generator."""
import numpy as np
import pytest
import torch

import synth
from oracle import reference as ref


def test_generators_are_deterministic():
    sh = synth.tiny_shape(d=32, hq=4, hkv=2, dh=8, f=16)
    a, b = synth.layer_weights(sh, 0, 3), synth.layer_weights(sh, 0, 3)
    for n in synth.WEIGHT_NAMES:
        assert np.array_equal(a[n][0], b[n][0]) and np.array_equal(a[n][1], b[n][1])
    c = synth.layer_weights(sh, 1, 3)
    assert not np.array_equal(a["wq"][0], c["wq"][0])
    k1, v1 = synth.kv_prior(sh, 0, 2, 5, 9)
    k2, v2 = synth.kv_prior(sh, 0, 2, 5, 9)
    assert np.array_equal(k1, k2) and np.array_equal(v1, v2)
    assert np.array_equal(synth.activations(3, 32), synth.activations(3, 32))


def test_quantiser_closed_form_bounds():
    rng = np.random.default_rng(0)
    w = (rng.standard_normal((64, 300)) * 0.02).astype(np.float32)
    w[5] = 0.0                                      # an all-zero row gets scale 1
    q, s = synth.quantize_rows(w)
    assert q.dtype == np.int8 and s.dtype == np.float32
    assert s[5] == 1.0 and not q[5].any()
    nz = np.arange(64) != 5
    assert np.all(np.abs(q[nz]).max(axis=1) == 127)           # the row maximum maps to +-127
    assert np.abs(q).max() <= 127                                # -128 is never used
    err = np.abs(w.astype(np.float64) - q.astype(np.float64) * s[:, None].astype(np.float64))
    assert np.all(err <= s[:, None].astype(np.float64) * 0.5 * (1 + 1e-6))


def test_bf16_rounding_matches_torch():
    rng = np.random.default_rng(1)
    a = np.concatenate([rng.standard_normal(10000).astype(np.float32) * 10.0 ** rng.integers(-8, 8, 10000),
                        np.array([0.0, -0.0, 1.0, 1.00390625, 1.01171875, -3.0e38], np.float32)])
    mine = synth.bf16_round(a)
    t = torch.from_numpy(a.copy()).to(torch.bfloat16).to(torch.float32).numpy()
    assert np.array_equal(mine, t)
    # the oracle's storage rounding (float64 -> 8 significant bits) agrees for float32 inputs
    assert np.array_equal(ref.bf16_store(a.astype(np.float64)).astype(np.float32), t)
    assert np.isnan(synth.bf16_round(np.array([np.nan], np.float32))[0])


def test_tiny_mask_recipe():
    q, kv, f = synth.tiny_mask(synth.TINY)
    assert q.sum() == 6 and kv.sum() == 2 and f.sum() == 1024
    qc, kvc, fc = ref.close_mask(q, kv, f, synth.TINY.group_size)
    assert np.array_equal(qc, q.astype(bool)) and kvc.all()


@pytest.mark.parametrize("seed", [1, 2, 3, 4, 5])
def test_budget_mask_hits_target(seed):
    sh = synth.LLAMA3_8B.with_layers(1, vocab=0)
    q, kv, f = synth.budget_mask(sh, seed)
    qc, kvc, fc = ref.close_mask(q, kv, f, sh.group_size)
    # closed by construction
    assert np.array_equal(qc, q.astype(bool)) and np.array_equal(kvc, kv.astype(bool))
    counts = synth.mask_counts(qc, kvc, fc)
    ratio = ref.active_flop_ratio(sh, counts)
    granule = 6 * sh.d_model * 128 / ref.layer_flops(sh, sh.n_q_heads, sh.n_kv_heads, sh.d_ffn)
    assert 0.57 - granule < ratio <= 0.57 + 1e-12
    assert counts[0][0] < sh.n_q_heads and counts[2][0] < sh.d_ffn


def test_budget_mask_stack_and_70b():
    for sh in (synth.LLAMA3_8B, synth.LLAMA3_70B):
        q, kv, f = synth.budget_mask(sh, 1)
        counts = synth.mask_counts(*ref.close_mask(q, kv, f, sh.group_size))
        assert abs(ref.active_flop_ratio(sh, counts) - 0.57) < 1e-3
