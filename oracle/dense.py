"""Third CPU reference: a textbook dense Llama decoder layer with no mask logic at all.

TEST INFRASTRUCTURE ONLY (see ``oracle.reference``). Written independently of the oracle's
zero-mask path: key/value heads are expanded to the query heads before a batched product, and
the rotary embedding is a complex rotation (pair (i, i + d_h/2) as real and imaginary parts).
Used for the invariant "all-kept mask == dense layer".
"""
from __future__ import annotations

import numpy as np

__all__ = ["dense_decode_layer"]


def _rms(v, g, eps):
    return v * (1.0 / np.sqrt((v ** 2).mean(-1, keepdims=True) + eps)) * g


def _rotate(x, pos, theta):
    half = x.shape[-1] // 2
    freq = np.exp(-np.log(theta) * 2.0 * np.arange(half) / x.shape[-1])
    z = (x[..., :half] + 1j * x[..., half:]) * np.exp(1j * pos * freq)
    return np.concatenate([z.real, z.imag], axis=-1)


def _bf16(a):
    m, e = np.frexp(a)
    return np.ldexp(np.rint(m * 256.0), e - 8)


def dense_decode_layer(Wd, x, k_cache, v_cache, pos, sh, round_cache=True):
    """``Wd`` holds float64 dense matrices wq..wd and gains attn_norm / ffn_norm."""
    Hq, Hkv, dh = sh.n_q_heads, sh.n_kv_heads, sh.head_dim
    rep = Hq // Hkv
    outs = []
    for b in range(x.shape[0]):
        h0 = np.asarray(x[b], np.float64)
        a = _rms(h0, Wd["attn_norm"], sh.rms_eps)
        q = _rotate((Wd["wq"] @ a).reshape(Hq, dh), pos, sh.rope_theta)
        k = _rotate((Wd["wk"] @ a).reshape(Hkv, dh), pos, sh.rope_theta)
        v = (Wd["wv"] @ a).reshape(Hkv, dh)
        k_cache[b, :, pos] = _bf16(k) if round_cache else k
        v_cache[b, :, pos] = _bf16(v) if round_cache else v
        Kx = np.repeat(k_cache[b, :, :pos + 1], rep, axis=0)       # [H_q][n][d_h]
        Vx = np.repeat(v_cache[b, :, :pos + 1], rep, axis=0)
        sc = np.einsum("hd,hnd->hn", q, Kx) / np.sqrt(dh)
        sc = np.exp(sc - sc.max(-1, keepdims=True))
        sc /= sc.sum(-1, keepdims=True)
        att = np.einsum("hn,hnd->hd", sc, Vx).reshape(-1)
        h1 = h0 + Wd["wo"] @ att
        f = _rms(h1, Wd["ffn_norm"], sh.rms_eps)
        gt = Wd["wg"] @ f
        outs.append(h1 + Wd["wd"] @ ((gt / (1.0 + np.exp(-gt))) * (Wd["wu"] @ f)))
    return np.stack(outs)
