"""Pins of the groupwise INT8 store format (one BF16 scale per output row and run of 128 input
columns) in the oracle's dequantisation and the synthetic quantiser."""
import numpy as np

import synth
from oracle import reference as ref


def test_dequantize_groupwise_hand_example():
    q = np.array([[1, -2, 3, 4], [5, 6, -7, 8]], np.int8)
    s = synth.to_bf16_bits(np.array([[0.5, 2.0], [1.0, 0.25]], np.float32))
    want = np.array([[0.5, -1.0, 6.0, 8.0], [5.0, 6.0, -1.75, 2.0]])
    assert np.array_equal(ref.dequantize(q, s), want)


def test_dequantize_groupwise_brute_force():
    rng = np.random.default_rng(3)
    q = rng.integers(-127, 128, (5, 384)).astype(np.int8)
    sv = synth.bf16_round(rng.uniform(1e-4, 1e-2, (5, 3)).astype(np.float32))
    got = ref.dequantize(q, synth.to_bf16_bits(sv))
    for o in range(5):
        for i in range(0, 384, 37):
            assert got[o, i] == float(q[o, i]) * float(sv[o, i // 128])


def test_equal_group_scales_equal_row_scales():
    """A groupwise store whose group scales all equal the row's BF16 scale dequantises to the
    per-row store exactly (the one-store validation's pair of identical quantisations)."""
    w = np.random.default_rng(4).standard_normal((64, 512)).astype(np.float32) * 0.02
    q, s = synth.quantize_rows_bf16(w)
    assert np.array_equal(synth.bf16_round(s), s)
    bits = np.repeat(synth.to_bf16_bits(s)[:, None], 512 // 128, axis=1)
    assert np.array_equal(ref.dequantize(q, bits), ref.dequantize(q, s))


def test_groupwise_quantiser_bounds():
    rng = np.random.default_rng(5)
    w = (rng.standard_normal((32, 1024)) * rng.uniform(0.001, 0.1, (32, 1))).astype(np.float32)
    w[3, 128:256] = 0.0                               # an all-zero group
    q, bits = synth.quantize_groups(w)
    s = synth.bf16_bits_to_f32(bits).astype(np.float64)
    assert q.dtype == np.int8 and np.abs(q.astype(int)).max() <= 127
    assert s.shape == (32, 8) and s[3, 1] == 1.0 and not q[3, 128:256].any()
    err = np.abs(w.astype(np.float64) - ref.dequantize(q, bits))
    amax = np.abs(w.reshape(32, 8, 128)).max(axis=2)
    # rounding error of at most half a step, or the clipping of a scale rounded down
    bound = np.maximum(s / 2, amax * 2.0 ** -8) * (1 + 1e-12)
    assert np.all(err.reshape(32, 8, 128) <= bound[:, :, None])
    # every non-zero group uses its full range
    big = np.abs(q.reshape(32, 8, 128).astype(int)).max(axis=2)
    assert np.all((big >= 126) | (amax == 0))


def test_groupwise_layer_same_draws():
    """The three quantisations come from the same float weights: they agree to within their
    quantisation steps."""
    sh = synth.tiny_shape(d=256, hq=4, hkv=2, dh=64, f=512, layers=1)
    a = synth.layer_weights(sh, 0, quant="group")
    b = synth.layer_weights(sh, 0)
    for n in ("wq", "wo", "wd"):
        da, db = ref.dequantize(*a[n]), ref.dequantize(*b[n])
        step = float(np.max(b[n][1]))
        assert np.abs(da - db).max() <= step
    assert np.array_equal(a["attn_norm"], b["attn_norm"])


def test_groupwise_decode_layer_matches_per_row_when_scales_agree():
    """decode_layer over a groupwise store with per-row-equal group scales equals decode_layer
    over the per-row store of the same bytes, bit for bit."""
    sh = synth.tiny_shape(d=256, hq=4, hkv=2, dh=64, f=512, layers=1)
    lw = synth.layer_weights(sh, 0, quant="row_bf16")
    gw = dict(lw)
    for n in ("wq", "wk", "wv", "wo", "wg", "wu", "wd"):
        q, s = lw[n]
        gw[n] = (q, np.repeat(synth.to_bf16_bits(s)[:, None], q.shape[1] // 128, axis=1))
    mask = ref.close_mask(*synth.tiny_mask(sh), sh.group_size)
    x = synth.activations(1, sh.d_model).astype(np.float64)
    outs = []
    for layer in (lw, gw):
        W = ref.masked_layer(layer, mask[0][0], mask[1][0], mask[2][0], sh.head_dim)
        K = np.zeros((1, sh.n_kv_heads, 8, sh.head_dim))
        V = np.zeros_like(K)
        outs.append(ref.decode_layer(W, x, K, V, 0, sh))
    assert np.array_equal(outs[0], outs[1])
