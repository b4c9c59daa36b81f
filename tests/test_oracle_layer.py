"""Whole-layer pins for the oracle.

* transformers' LlamaDecoderLayer (a third-party implementation, float64) for the dense layer,
  for decode against a prior cache and for causal prefill;
* structural removal: a mask that drops whole KV groups or FFN channels equals a smaller
  transformers layer holding only the retained slices;
* weights of dropped modules do not influence the output, retained ones do;
* pure-Python scalar loops on a tiny layer; the compacted-panel reference (mask-as-zero
  control, Table "systems"); the textbook dense layer for the all-kept mask;
* batch rows are independent; prefill equals sequential decode; empty modules.
"""
import numpy as np
import pytest

import synth
from oracle import compact, dense, reference as ref, scalar
from tests.helpers import caches_f64, hf_decode, hf_prefill, make_store

IDENT = lambda a: np.asarray(a, np.float64)  # noqa: E731   cache storage without rounding

SMALL = synth.tiny_shape(d=64, hq=8, hkv=2, dh=16, f=96, theta=10000.0)


def _masked(sh, layer, mask):
    qc, kvc, fc = ref.close_mask(*mask, sh.group_size)
    return ref.masked_layer(layer, qc[0], kvc[0], fc[0], sh.head_dim), (qc, kvc, fc)


def test_dense_decode_matches_transformers():
    sh, pos = SMALL, 11
    layer = make_store(sh)[0]
    W, _ = _masked(sh, layer, synth.all_kept_mask(sh))
    x = synth.activations(1, sh.d_model)
    (K, V), = caches_f64(sh, 1, pos, pos + 1)
    kp, vp = K[0, :, :pos].copy(), V[0, :, :pos].copy()
    out = ref.decode_layer(W, x, K, V, pos, sh, kv_store=IDENT)[0]
    hf = hf_decode(sh, W, x[0], kp, vp, pos)
    assert np.allclose(out, hf, rtol=0, atol=2e-6 * np.abs(hf).max())


def test_dense_prefill_matches_transformers():
    sh, T = SMALL, 9
    layer = make_store(sh)[0]
    W, _ = _masked(sh, layer, synth.all_kept_mask(sh))
    x = synth.activations(T, sh.d_model)
    K = np.zeros((sh.n_kv_heads, T, sh.head_dim))
    V = np.zeros_like(K)
    out = ref.prefill_layer(W, x, K, V, 0, sh, kv_store=IDENT)
    hf = hf_prefill(sh, W, x)
    assert np.allclose(out, hf, rtol=0, atol=2e-6 * np.abs(hf).max())


def test_structural_removal_matches_smaller_transformers_layer():
    """Dropping KV group 1 (with its heads) and 40 FFN channels is the same computation as a
    Llama layer that never had them."""
    sh, pos = SMALL, 6
    layer = make_store(sh)[0]
    q, kv, f = synth.all_kept_mask(sh)
    kv[0, 1] = 0
    rng = np.random.default_rng(9)
    f[0, rng.choice(sh.d_ffn, 40, replace=False)] = 0
    W, (qc, kvc, fc) = _masked(sh, layer, (q, kv, f))
    x = synth.activations(1, sh.d_model)
    (K, V), = caches_f64(sh, 1, pos, pos + 1)
    kp, vp = K[0, :1, :pos].copy(), V[0, :1, :pos].copy()
    out = ref.decode_layer(W, x, K, V, pos, sh, kv_store=IDENT)[0]

    dh, keep_ch = sh.head_dim, np.flatnonzero(fc[0])
    full = {n: ref.dequantize(*layer[n]) for n in synth.WEIGHT_NAMES}
    rows_q = np.arange(0, 4 * dh)                       # heads 0..3 of group 0
    small = {"wq": full["wq"][rows_q], "wk": full["wk"][:dh], "wv": full["wv"][:dh],
             "wo": full["wo"][:, rows_q], "wg": full["wg"][keep_ch], "wu": full["wu"][keep_ch],
             "wd": full["wd"][:, keep_ch], "attn_norm": W["attn_norm"], "ffn_norm": W["ffn_norm"]}
    hf = hf_decode(sh, small, x[0], kp, vp, pos)
    assert np.allclose(out, hf, rtol=0, atol=2e-6 * np.abs(hf).max())


def test_dropped_weights_have_no_influence_and_kept_ones_do():
    sh, pos = SMALL, 5
    layer = make_store(sh)[0]
    q, kv, f = synth.all_kept_mask(sh)
    q[0, [1, 6]] = 0                 # one head dropped inside each group
    f[0, ::3] = 0
    x = synth.activations(2, sh.d_model)

    def run(lay):
        W, _ = _masked(sh, lay, (q, kv, f))
        caches = caches_f64(sh, 2, pos, pos + 1)
        return ref.decode_layer(W, x, caches[0][0], caches[0][1], pos, sh)

    base = run(layer)
    dh = sh.head_dim
    noisy = {k: (v[0].copy(), v[1].copy()) if isinstance(v, tuple) else v for k, v in layer.items()}
    rng = np.random.default_rng(3)
    for h in (1, 6):
        noisy["wq"][0][h * dh:(h + 1) * dh] = rng.integers(-127, 128, (dh, sh.d_model))
        noisy["wo"][0][:, h * dh:(h + 1) * dh] = rng.integers(-127, 128, (sh.d_model, dh))
    for name in ("wg", "wu"):
        noisy[name][0][::3] = rng.integers(-127, 128, noisy[name][0][::3].shape)
    noisy["wd"][0][:, ::3] = rng.integers(-127, 128, noisy["wd"][0][:, ::3].shape)
    assert np.array_equal(run(noisy), base)
    for name, sl in (("wq", np.s_[0:1]), ("wo", np.s_[:, 0:1]), ("wk", np.s_[0:1]),
                     ("wg", np.s_[1:2]), ("wd", np.s_[:, 1:2])):
        alt = {k: (v[0].copy(), v[1]) if isinstance(v, tuple) else v for k, v in layer.items()}
        alt[name][0][sl] = -alt[name][0][sl] - 1
        assert not np.allclose(run(alt), base, rtol=0, atol=1e-9), name


def _scalar_layer(layer):
    conv = {}
    for n in synth.WEIGHT_NAMES:
        conv[n] = (layer[n][0].astype(int).tolist(), layer[n][1].astype(float).tolist())
    conv["attn_norm"] = ref.bf16_bits_to_f64(layer["attn_norm"]).tolist()
    conv["ffn_norm"] = ref.bf16_bits_to_f64(layer["ffn_norm"]).tolist()
    return conv


@pytest.mark.parametrize("seed", range(6))
def test_scalar_brute_force(seed):
    sh, pos = synth.tiny_shape(d=16, hq=4, hkv=2, dh=4, f=8), 3
    layer = make_store(sh, seed_w=seed)[0]
    mask = synth.raw_mask(sh, seed, p_q=0.6, p_kv=0.8, p_f=0.6) if seed else synth.all_kept_mask(sh)
    W, (qc, kvc, fc) = _masked(sh, layer, mask)
    x = synth.activations(1, sh.d_model, seed_x=seed + 10)
    (K, V), = caches_f64(sh, 1, pos, pos + 1, seed_kv=seed)
    kc, vc = K[0].tolist(), V[0].tolist()
    out = ref.decode_layer(W, x, K, V, pos, sh)[0]
    got = scalar.scalar_decode_layer(_scalar_layer(layer), qc[0].tolist(), kvc[0].tolist(),
                                     fc[0].tolist(), x[0].tolist(), kc, vc, pos, sh)
    assert np.allclose(got, out, rtol=1e-12, atol=1e-12)
    for g in np.flatnonzero(kvc[0]):                    # retained groups' cache rows agree
        assert np.allclose(np.array(kc)[g, pos], K[0, g, pos], rtol=0, atol=0)


def test_compacted_equals_zero_masked_sweep():
    """Mask-as-zero control: packing changes nothing but speed. All 2^4 x 2^2 head/group masks
    times several FFN masks on a tiny layer, closed first."""
    sh, pos = synth.tiny_shape(d=16, hq=4, hkv=2, dh=4, f=8), 4
    layer = make_store(sh)[0]
    x = synth.activations(2, sh.d_model)
    rng = np.random.default_rng(0)
    for qv in range(16):
        for kvv in range(4):
            fbits = rng.integers(0, 2, (1, 8)).astype(np.uint8)
            q = np.array([[(qv >> i) & 1 for i in range(4)]], np.uint8)
            kv = np.array([[(kvv >> i) & 1 for i in range(2)]], np.uint8)
            W, (qc, kvc, fc) = _masked(sh, layer, (q, kv, fbits))
            c1 = caches_f64(sh, 2, pos, pos + 1)
            c2 = caches_f64(sh, 2, pos, pos + 1)
            a = ref.decode_layer(W, x, c1[0][0], c1[0][1], pos, sh)
            pn = compact.compact_panels(layer, qc[0], kvc[0], fc[0], sh)
            b = compact.compact_decode_layer(pn, x, c2[0][0], c2[0][1], pos, sh)
            assert np.allclose(a, b, rtol=1e-12, atol=1e-12)


def test_zeroed_store_is_the_zero_masked_layer():
    """The store of the mask-as-zero control (dropped modules' INT8 weights zeroed, scales kept),
    read as a dense layer, dequantises to the oracle's zero-masked layer and decodes to the same
    output as the masked layer."""
    sh, pos = SMALL, 128
    layer = make_store(sh)[0]
    mask = synth.raw_mask(sh, 5)
    W, (qc, kvc, fc) = _masked(sh, layer, mask)
    z = synth.zero_dropped(layer, sh, qc[0], kvc[0], fc[0])
    Wz, _ = _masked(sh, z, synth.all_kept_mask(sh))
    for name in W:
        assert np.array_equal(W[name], Wz[name]), name
    x = synth.activations(1, sh.d_model)
    c1 = caches_f64(sh, 1, pos, pos + 1)
    c2 = caches_f64(sh, 1, pos, pos + 1)
    a = ref.decode_layer(W, x, c1[0][0], c1[0][1], pos, sh)
    b = ref.decode_layer(Wz, x, c2[0][0], c2[0][1], pos, sh)
    assert np.array_equal(a, b)


@pytest.mark.parametrize("sh", [SMALL, synth.TINY], ids=["small", "tiny_cfg"])
def test_compacted_equals_zero_masked_configs(sh):
    pos = 128
    layer = make_store(sh)[0]
    mask = synth.tiny_mask(sh) if sh is synth.TINY else synth.raw_mask(sh, 4)
    W, (qc, kvc, fc) = _masked(sh, layer, mask)
    x = synth.activations(1, sh.d_model)
    c1 = caches_f64(sh, 1, pos, pos + 1)
    c2 = caches_f64(sh, 1, pos, pos + 1)
    a = ref.decode_layer(W, x, c1[0][0], c1[0][1], pos, sh)
    pn = compact.compact_panels(layer, qc[0], kvc[0], fc[0], sh)
    b = compact.compact_decode_layer(pn, x, c2[0][0], c2[0][1], pos, sh)
    m, s = np.abs(a - b).max() / np.abs(a).max(), np.abs(a - b).sum() / np.abs(a).sum()
    assert m < 1e-12 and s < 1e-12


def test_all_kept_equals_textbook_dense():
    sh, pos = synth.TINY, 128
    layer = make_store(sh)[0]
    W, _ = _masked(sh, layer, synth.all_kept_mask(sh))
    x = synth.activations(1, sh.d_model)
    c1 = caches_f64(sh, 1, pos, pos + 1)
    c2 = caches_f64(sh, 1, pos, pos + 1)
    a = ref.decode_layer(W, x, c1[0][0], c1[0][1], pos, sh)
    b = dense.dense_decode_layer(W, x, c2[0][0], c2[0][1], pos, sh)
    assert np.allclose(a, b, rtol=1e-12, atol=1e-12)
    assert np.array_equal(c1[0][0][:, :, pos], c2[0][0][:, :, pos])


def test_empty_modules():
    sh, pos = SMALL, 3
    layer = make_store(sh)[0]
    x = synth.activations(1, sh.d_model)
    q, kv, f = synth.all_kept_mask(sh)
    W, _ = _masked(sh, layer, (q * 0, kv, f * 0))          # nothing retained: identity layer
    (K, V), = caches_f64(sh, 1, pos, pos + 1)
    assert np.array_equal(ref.decode_layer(W, x, K, V, pos, sh), x.astype(np.float64))
    # attention fully dropped: the FFN sees the input residual (transformers' MLP + RMSNorm)
    import torch
    from transformers.models.llama.modeling_llama import LlamaMLP, LlamaRMSNorm
    from transformers import LlamaConfig
    W, _ = _masked(sh, layer, (q * 0, kv, f))
    (K, V), = caches_f64(sh, 1, pos, pos + 1)
    out = ref.decode_layer(W, x, K, V, pos, sh)[0]
    cfg = LlamaConfig(hidden_size=sh.d_model, intermediate_size=sh.d_ffn, mlp_bias=False,
                      rms_norm_eps=sh.rms_eps)
    mlp, nrm = LlamaMLP(cfg).double(), LlamaRMSNorm(sh.d_model, sh.rms_eps).double()
    with torch.no_grad():
        for mod, name in ((mlp.gate_proj, "wg"), (mlp.up_proj, "wu"), (mlp.down_proj, "wd")):
            mod.weight.copy_(torch.tensor(W[name]))
        nrm.weight.copy_(torch.tensor(W["ffn_norm"]))
        xt = torch.tensor(x[0], dtype=torch.float64)
        lib = (xt + mlp(nrm(xt))).numpy()
    assert np.allclose(out, lib, rtol=0, atol=1e-6 * np.abs(lib).max())


def test_batch_rows_are_independent():
    sh, pos, B = SMALL, 7, 4
    layer = make_store(sh)[0]
    W, _ = _masked(sh, layer, synth.raw_mask(sh, 2))
    x = synth.activations(B, sh.d_model)
    (K, V), = caches_f64(sh, B, pos, pos + 1)
    full = ref.decode_layer(W, x, K.copy(), V.copy(), pos, sh)
    for b in range(B):
        one = ref.decode_layer(W, x[b:b + 1], K[b:b + 1].copy(), V[b:b + 1].copy(), pos, sh)
        assert np.array_equal(one[0], full[b])


@pytest.mark.parametrize("pos0", [0, 5])
def test_prefill_equals_sequential_decode(pos0):
    sh, T = SMALL, 6
    layer = make_store(sh)[0]
    W, _ = _masked(sh, layer, synth.raw_mask(sh, 1))
    x = synth.activations(T, sh.d_model)
    (K, V), = caches_f64(sh, 1, pos0, pos0 + T)
    Kp, Vp = K[0].copy(), V[0].copy()
    pre = ref.prefill_layer(W, x, Kp, Vp, pos0, sh)
    seq = np.stack([ref.decode_layer(W, x[t:t + 1], K, V, pos0 + t, sh)[0] for t in range(T)])
    assert np.allclose(pre, seq, rtol=1e-12, atol=1e-12)
    assert np.array_equal(Kp, K[0]) and np.array_equal(Vp, V[0])


def test_stack_logits_match_transformers_model():
    import torch
    from transformers import LlamaConfig, LlamaForCausalLM
    sh = synth.tiny_shape(d=32, hq=4, hkv=2, dh=8, f=48, layers=2, vocab=50, theta=10000.0)
    store = make_store(sh)
    fn, lm = synth.final_norm(sh), synth.lm_head(sh)
    T = 5
    x = synth.activations(T, sh.d_model)
    mask = ref.close_mask(*synth.all_kept_mask(sh), sh.group_size)
    caches = [(np.zeros((sh.n_kv_heads, T, sh.head_dim)),) * 1 + (np.zeros((sh.n_kv_heads, T, sh.head_dim)),)
              for _ in range(sh.n_layers)]
    logits = ref.prefill_stack(lambda l: store[l], mask, x, caches, 0, sh, fn, lm, kv_store=IDENT)

    cfg = LlamaConfig(hidden_size=sh.d_model, intermediate_size=sh.d_ffn, num_attention_heads=sh.n_q_heads,
                      num_key_value_heads=sh.n_kv_heads, head_dim=sh.head_dim, num_hidden_layers=2,
                      vocab_size=sh.vocab, rms_norm_eps=sh.rms_eps, tie_word_embeddings=False,
                      rope_parameters={"rope_type": "default", "rope_theta": sh.rope_theta})
    cfg._attn_implementation = "eager"
    model = LlamaForCausalLM(cfg).double().eval()
    names = {"wq": "self_attn.q_proj", "wk": "self_attn.k_proj", "wv": "self_attn.v_proj",
             "wo": "self_attn.o_proj", "wg": "mlp.gate_proj", "wu": "mlp.up_proj", "wd": "mlp.down_proj"}
    with torch.no_grad():
        for l, lay in enumerate(store):
            mod = model.model.layers[l]
            for k, path in names.items():
                mod.get_submodule(path).weight.copy_(torch.tensor(ref.dequantize(*lay[k])))
            mod.input_layernorm.weight.copy_(torch.tensor(ref.bf16_bits_to_f64(lay["attn_norm"])))
            mod.post_attention_layernorm.weight.copy_(torch.tensor(ref.bf16_bits_to_f64(lay["ffn_norm"])))
        model.model.norm.weight.copy_(torch.tensor(ref.bf16_bits_to_f64(fn)))
        model.lm_head.weight.copy_(torch.tensor(ref.bf16_bits_to_f64(lm)))
        hf = model(inputs_embeds=torch.tensor(x, dtype=torch.float64)[None]).logits[0].numpy()
    assert np.allclose(logits, hf, rtol=0, atol=5e-6 * np.abs(hf).max())
