"""Pins for the oracle's building blocks against closed forms and library routines."""
import math

import numpy as np
import pytest
import torch
import torch.nn.functional as Fn

from oracle import reference as ref


def test_rmsnorm_closed_form_and_library():
    rng = np.random.default_rng(0)
    r = rng.standard_normal((5, 64)) * 3.0
    eps = 1e-5
    n = ref.rms_norm(r, np.ones(64), eps)
    ms = (r * r).mean(axis=1)
    assert np.allclose((n * n).mean(axis=1), ms / (ms + eps), rtol=1e-13, atol=0)
    g = rng.standard_normal(64)
    lib = Fn.rms_norm(torch.tensor(r), (64,), weight=torch.tensor(g), eps=eps).numpy()
    assert np.allclose(ref.rms_norm(r, g, eps), lib, rtol=1e-12, atol=1e-14)


def test_rope_special_angles_pin_rotate_half():
    # d_h = 4: pairs (0, 2) and (1, 3); inv_freq = [1, theta^-1/2]. With theta = (2 pos / pi)^2
    # the second pair turns by exactly pi/2 and the first by pos radians.
    pos = 3
    theta = (2.0 * pos / math.pi) ** 2
    x = np.array([[[1.0, 2.0, 3.0, 4.0]]])
    y = ref.rope(x, [pos], theta)[0, 0]
    c, s = math.cos(pos), math.sin(pos)
    expect = [1.0 * c - 3.0 * s, -4.0, 3.0 * c + 1.0 * s, 2.0]
    assert np.allclose(y, expect, rtol=0, atol=1e-12)


def test_rope_invariants():
    rng = np.random.default_rng(1)
    dh, theta = 64, 500000.0
    x = rng.standard_normal((3, 1, dh))
    assert np.array_equal(ref.rope(x, [0], theta), x)                      # pos 0 is identity
    y = ref.rope(x, [1234], theta)
    half = dh // 2
    pair_norm = lambda a: a[..., :half] ** 2 + a[..., half:] ** 2         # noqa: E731
    assert np.allclose(pair_norm(y), pair_norm(x), rtol=1e-12)
    # relative position: <R(p) q, R(p') k> depends on p - p' only
    q, k = rng.standard_normal((1, 1, dh)), rng.standard_normal((1, 1, dh))
    a = (ref.rope(q, [100], theta) * ref.rope(k, [40], theta)).sum()
    b = (ref.rope(q, [1060], theta) * ref.rope(k, [1000], theta)).sum()
    assert abs(a - b) < 1e-10


def test_rope_matches_transformers():
    from transformers.models.llama.modeling_llama import apply_rotary_pos_emb
    rng = np.random.default_rng(2)
    dh, theta, pos = 128, 500000.0, np.array([0, 7, 2048, 8191])
    q = rng.standard_normal((1, 2, 4, dh))
    k = rng.standard_normal((1, 1, 4, dh))
    # cos/sin built in float64 from the same angle definition (angles are the paper-free input)
    inv = 1.0 / (theta ** (np.arange(0, dh, 2) / dh))
    ang = np.concatenate([pos[:, None] * inv, pos[:, None] * inv], axis=1)[None]
    qe, ke = apply_rotary_pos_emb(torch.tensor(q), torch.tensor(k), torch.tensor(np.cos(ang)),
                                  torch.tensor(np.sin(ang)))
    assert np.allclose(ref.rope(q[0], pos, theta), qe.numpy()[0], rtol=0, atol=1e-12)
    assert np.allclose(ref.rope(k[0], pos, theta), ke.numpy()[0], rtol=0, atol=1e-12)


def test_softmax_rows():
    rng = np.random.default_rng(3)
    s = rng.standard_normal((7, 300)) * 20
    p = ref.softmax(s)
    assert np.all(p >= 0) and np.allclose(p.sum(axis=1), 1.0, rtol=0, atol=1e-12)
    assert np.allclose(p, torch.softmax(torch.tensor(s), -1).numpy(), rtol=1e-12, atol=1e-15)


def test_silu_library():
    z = np.linspace(-30, 30, 1001)
    assert np.allclose(ref.silu(z), Fn.silu(torch.tensor(z)).numpy(), rtol=1e-13, atol=1e-300)


@pytest.mark.parametrize("causal", [False, True])
def test_gqa_attention_matches_sdpa(causal):
    rng = np.random.default_rng(4)
    Hq, Hkv, T, n, dh = 8, 2, 5, 37, 16
    q = rng.standard_normal((Hq, T, dh))
    K, V = rng.standard_normal((Hkv, n, dh)), rng.standard_normal((Hkv, n, dh))
    off = n - T if causal else None
    o = ref.gqa_attention(q, K, V, Hq // Hkv, causal_offset=off)
    mask = None
    if causal:
        mask = torch.tensor(np.arange(n)[None, :] <= (off + np.arange(T))[:, None])
    lib = Fn.scaled_dot_product_attention(torch.tensor(q)[None], torch.tensor(K)[None],
                                          torch.tensor(V)[None], attn_mask=mask,
                                          enable_gqa=True)[0].numpy()
    assert np.allclose(o, lib, rtol=1e-12, atol=1e-13)


def test_attention_special_cases():
    rng = np.random.default_rng(5)
    dh = 8
    q = rng.standard_normal((4, 1, dh))
    k_row = rng.standard_normal(dh)
    K = np.tile(k_row, (2, 9, 1))                     # identical keys -> uniform weights
    V = rng.standard_normal((2, 9, dh))
    o = ref.gqa_attention(q, K, V, 2)
    assert np.allclose(o[0, 0], V[0].mean(axis=0), rtol=1e-12)
    assert np.allclose(o[3, 0], V[1].mean(axis=0), rtol=1e-12)
    one = ref.gqa_attention(q, K[:, :1], V[:, :1], 2)   # a single position returns its value
    assert np.allclose(one[1, 0], V[0, 0]) and np.allclose(one[2, 0], V[1, 0])
