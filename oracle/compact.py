"""Second CPU reference: the layer computed from physically compacted INT8 panels.

TEST INFRASTRUCTURE ONLY (see ``oracle.reference``). Used for two invariants:
* the compacted computation equals the zero-masked oracle (the paper's mask-as-zero control,
  Table "systems": packing changes speed, not results);
* byte-exact comparison of the panels a compiled plan holds.

Panels ("Backing-store semantics" paragraph: contiguous retained-coordinate tensors), all
int8 row-major ``[out][in]`` with float32 per-row scales:
* QKV: rows of the retained query heads (ascending), then K rows and V rows of the retained
  KV groups (ascending); scales move with their rows;
* O: the columns of W_o belonging to retained query heads; all d scales unchanged;
* gate, up: rows of the retained channels; scales move with their rows;
* down: the columns of W_down of the retained channels; all d scales unchanged.
The output of a panel product is s * (P x): dequantisation after the integer-weight dot product.
"""
from __future__ import annotations

import numpy as np

from .reference import (bf16_bits_to_f64, bf16_store, index_lists, rms_norm, rope, silu,
                        softmax)

__all__ = ["compact_panels", "compact_decode_layer"]


def _head_rows(idx, dh):
    if len(idx) == 0:
        return np.zeros(0, dtype=np.int64)
    return (np.asarray(idx, dtype=np.int64)[:, None] * dh + np.arange(dh)[None, :]).ravel()


def compact_panels(layer, qc_l, kvc_l, ffnc_l, sh):
    dh = sh.head_dim
    q_idx, kv_idx, q_kvslot, ffn_idx = index_lists(qc_l, kvc_l, ffnc_l, sh.group_size)
    rq, rkv = _head_rows(q_idx, dh), _head_rows(kv_idx, dh)
    wq, sq = layer["wq"]
    wk, sk = layer["wk"]
    wv, sv = layer["wv"]
    wo, so = layer["wo"]
    wg, sg = layer["wg"]
    wu, su = layer["wu"]
    wd, sd = layer["wd"]
    return {
        "q_idx": q_idx, "kv_idx": kv_idx, "q_kvslot": q_kvslot, "ffn_idx": ffn_idx,
        "qkv": np.concatenate([wq[rq], wk[rkv], wv[rkv]], axis=0),
        "qkv_scale": np.concatenate([sq[rq], sk[rkv], sv[rkv]]),
        "o": np.ascontiguousarray(wo[:, rq]), "o_scale": so.copy(),
        "gate": wg[ffn_idx], "gate_scale": sg[ffn_idx],
        "up": wu[ffn_idx], "up_scale": su[ffn_idx],
        "down": np.ascontiguousarray(wd[:, ffn_idx]), "down_scale": sd.copy(),
        "attn_norm": bf16_bits_to_f64(layer["attn_norm"]),
        "ffn_norm": bf16_bits_to_f64(layer["ffn_norm"]),
    }


def _panel_product(P, s, x):
    return np.asarray(s, np.float64) * (np.asarray(P, np.float64) @ x)


def compact_decode_layer(pn, x, k_cache, v_cache, pos, sh, kv_store=bf16_store):
    """Decode one layer from compacted panels. Only retained KV groups' cache rows are written;
    retained head i reads KV group kv_idx[q_kvslot[i]]."""
    dh = sh.head_dim
    m_q, m_kv = len(pn["q_idx"]), len(pn["kv_idx"])
    x = np.asarray(x, dtype=np.float64)
    out = np.empty_like(x)
    for b in range(x.shape[0]):
        r = x[b]
        n = rms_norm(r, pn["attn_norm"], sh.rms_eps)
        y = _panel_product(pn["qkv"], pn["qkv_scale"], n)
        q = y[:m_q * dh].reshape(m_q, 1, dh)
        k = y[m_q * dh:(m_q + m_kv) * dh].reshape(m_kv, 1, dh)
        v = y[(m_q + m_kv) * dh:].reshape(m_kv, 1, dh)
        q = rope(q, [pos], sh.rope_theta)[:, 0]
        k = rope(k, [pos], sh.rope_theta)[:, 0]
        for j, g in enumerate(pn["kv_idx"]):
            k_cache[b, g, pos] = kv_store(k[j])
            v_cache[b, g, pos] = kv_store(v[j, 0])
        o = np.zeros((m_q, dh))
        for i in range(m_q):
            g = pn["kv_idx"][pn["q_kvslot"][i]]
            p = softmax(k_cache[b, g, :pos + 1] @ q[i] / np.sqrt(dh))
            o[i] = p @ v_cache[b, g, :pos + 1]
        r = r + _panel_product(pn["o"], pn["o_scale"], o.reshape(-1))
        n2 = rms_norm(r, pn["ffn_norm"], sh.rms_eps)
        g_ = _panel_product(pn["gate"], pn["gate_scale"], n2)
        u_ = _panel_product(pn["up"], pn["up_scale"], n2)
        r = r + _panel_product(pn["down"], pn["down_scale"], silu(g_) * u_)
        out[b] = r
    return out
