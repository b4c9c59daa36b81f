"""Shared test utilities: error metrics, store builders and a third-party Llama layer."""
from __future__ import annotations

import numpy as np

import synth


def rel_errors(got, ref):
    """(max|err| / max|ref|, sum|err| / sum|ref|): the two parity metrics for floating point."""
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    err = np.abs(got - ref)
    return float(err.max() / np.abs(ref).max()), float(err.sum() / np.abs(ref).sum())


def assert_parity(got, ref, max_rel=1e-2, sum_rel=2e-3, what=""):
    """Floating-point parity bar: max|err| <= 1e-2 max|ref| and sum|err|/sum|ref| <= 2e-3."""
    assert np.all(np.isfinite(got)), f"{what}: non-finite output"
    m, s = rel_errors(got, ref)
    assert m <= max_rel and s <= sum_rel, f"{what}: max_rel={m:.3e} sum_rel={s:.3e}"
    return m, s


def make_store(sh, seed_w=0):
    return [synth.layer_weights(sh, l, seed_w) for l in range(sh.n_layers)]


def caches_f64(sh, batch, pos, max_seq, seed_kv=2):
    """Per-layer float64 (K, V) ``[B][H_kv][S][d_h]`` from the synthetic BF16 prior."""
    out = []
    for l in range(sh.n_layers):
        k, v = synth.kv_prior(sh, l, batch, pos, max_seq, seed_kv)
        out.append((synth.bf16_bits_to_f32(k).astype(np.float64),
                    synth.bf16_bits_to_f32(v).astype(np.float64)))
    return out


def hf_llama_layer(sh, Wd):
    """transformers' LlamaDecoderLayer in float64 holding the dense matrices ``Wd``."""
    import torch
    from transformers import LlamaConfig
    from transformers.models.llama.modeling_llama import LlamaDecoderLayer, LlamaRotaryEmbedding

    cfg = LlamaConfig(hidden_size=sh.d_model, intermediate_size=Wd["wg"].shape[0],
                      num_attention_heads=Wd["wq"].shape[0] // sh.head_dim,
                      num_key_value_heads=Wd["wk"].shape[0] // sh.head_dim,
                      head_dim=sh.head_dim, rms_norm_eps=sh.rms_eps,
                      rope_parameters={"rope_type": "default", "rope_theta": sh.rope_theta},
                      attention_bias=False, mlp_bias=False, max_position_embeddings=65536)
    cfg._attn_implementation = "eager"
    layer = LlamaDecoderLayer(cfg, layer_idx=0).double().eval()
    t = lambda a: torch.tensor(np.asarray(a), dtype=torch.float64)  # noqa: E731
    with torch.no_grad():
        layer.self_attn.q_proj.weight.copy_(t(Wd["wq"]))
        layer.self_attn.k_proj.weight.copy_(t(Wd["wk"]))
        layer.self_attn.v_proj.weight.copy_(t(Wd["wv"]))
        layer.self_attn.o_proj.weight.copy_(t(Wd["wo"]))
        layer.mlp.gate_proj.weight.copy_(t(Wd["wg"]))
        layer.mlp.up_proj.weight.copy_(t(Wd["wu"]))
        layer.mlp.down_proj.weight.copy_(t(Wd["wd"]))
        layer.input_layernorm.weight.copy_(t(Wd["attn_norm"]))
        layer.post_attention_layernorm.weight.copy_(t(Wd["ffn_norm"]))
    return layer, LlamaRotaryEmbedding(cfg), cfg


class PriorCache:
    """Minimal cache object for transformers' attention: prepends fixed prior keys/values."""

    def __init__(self, k, v):
        import torch
        self.k = torch.tensor(k, dtype=torch.float64)[None]
        self.v = torch.tensor(v, dtype=torch.float64)[None]

    def update(self, k, v, layer_idx, *a, **kw):
        import torch
        return torch.cat([self.k, k], dim=2), torch.cat([self.v, v], dim=2)


def hf_decode(sh, Wd, x_row, k_prior, v_prior, pos):
    """Decode one token at position ``pos`` with transformers, prior K/V ``[H_kv][pos][d_h]``."""
    import torch
    layer, rot, _ = hf_llama_layer(sh, Wd)
    h = torch.tensor(np.asarray(x_row), dtype=torch.float64)[None, None, :]
    pid = torch.tensor([[pos]])
    with torch.no_grad():
        cos, sin = rot(h, pid)
        out = layer(h, attention_mask=None, position_ids=pid,
                    past_key_values=PriorCache(k_prior, v_prior), position_embeddings=(cos, sin))
    return out[0, 0].numpy()


def hf_prefill(sh, Wd, x):
    """Causal prefill of ``x [T][d]`` from an empty cache with transformers."""
    import torch
    layer, rot, _ = hf_llama_layer(sh, Wd)
    T = x.shape[0]
    h = torch.tensor(np.asarray(x), dtype=torch.float64)[None]
    pid = torch.arange(T)[None]
    mask = torch.full((T, T), float("-inf"), dtype=torch.float64).triu(1)[None, None]
    with torch.no_grad():
        cos, sin = rot(h, pid)
        out = layer(h, attention_mask=mask, position_ids=pid, position_embeddings=(cos, sin))
    return out[0].numpy()


def teacher_forced_rows(layer_source, closed, table, scales, prompt, ids, sh, fn, lm):
    """The oracle's logits along a sequence whose generated part is given (teacher forcing):
    one prefill of prompt + ids[:-1] from an empty cache, which equals the oracle's request loop
    (pinned in tests/test_oracle_generate.py); row s holds the logits that chose ids[s]."""
    from oracle import reference as ref
    T = len(prompt)
    seq = np.concatenate([np.asarray(prompt), np.asarray(ids[:-1])]).astype(np.int64)
    S_ = len(seq)
    caches = [(np.zeros((sh.n_kv_heads, S_, sh.head_dim)), np.zeros((sh.n_kv_heads, S_, sh.head_dim)))
              for _ in range(sh.n_layers)]
    logits = ref.prefill_stack(layer_source, closed, ref.embed_rows(table, scales, seq), caches, 0,
                               sh, fn, lm)
    return logits[T - 1:]


def check_greedy_ids(ids, oracle_rows, what=""):
    """Greedy ids decided in floating point (several ids can be correct at a near tie): every
    step's id must be one whose oracle logit lies within the parity tolerance (1e-2 max|logit|)
    of the oracle's maximum, so a wrong id anywhere fails while a legitimate near tie passes.
    Returns the number of steps whose oracle decision was clear of the tolerance (those ids are
    then necessarily the oracle's argmax)."""
    clear = 0
    for s, (i, row) in enumerate(zip(ids, oracle_rows)):
        tol = 1e-2 * np.abs(row).max()
        assert row[i] >= row.max() - tol, \
            f"{what} step {s}: id {i} logit {row[i]:.6g} vs max {row.max():.6g} (tol {tol:.3g})"
        top2 = np.sort(row)[-2:]
        if top2[1] - top2[0] > tol:
            assert i == int(np.argmax(row))
            clear += 1
    return clear
