"""CPU oracle for a Llama-3-style decoder layer (and stack) run under one structured mask.

TEST INFRASTRUCTURE ONLY. Nothing on the product path imports, calls or links this module:
only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of ``bench.py`` do. It is
deliberately plain and slow: float64 numpy, dequantised weights, and the mask applied by zeroing
the masked modules in dense matrices (the paper's mask-as-zero control, Table "systems", which
holds the mask fixed and changes only physical packing). It shares no code with the HIP path;
inputs come from the ``synth`` generators.

Notation (paper, appendix "Candidate Construction, FLOP Ledger, and One-Store Validation"):
d model width, d_h head dimension, H_q / H_kv query and KV heads, d_f SwiGLU inner width,
m^q, m^kv, c the retained query heads, KV groups and SwiGLU channels of a layer.

Readings of points the paper leaves open (each is listed in the design notes):
* quantisation is symmetric INT8 with one float32 scale per output row; a layer's weight is
  W = q * s (q int8, s per row), and scales are never recomputed after masking; the groupwise
  store keeps one BF16 scale per output row and run of 128 input columns instead;
* query head h belongs to KV group g(h) = floor(h / r), r = H_q / H_kv (contiguous groups);
* closure: a head whose KV group is dropped is dropped; a KV group is kept iff any of its
  query heads is kept; FFN channels are kept as given (gate row, up row and down column move
  together);
* a dropped query head contributes nothing: its W_q rows and the matching W_o columns are zero;
* RoPE is rotate-half over pairs (i, i + d_h/2), angle pos * theta^(-2i/d_h), theta = 500000;
* RMSNorm: n = r / sqrt(mean(r^2) + eps) * gamma, eps = 1e-5;
* SwiGLU: h = silu(W_gate n) * (W_up n), silu(z) = z / (1 + exp(-z));
* the KV cache stores BF16 post-RoPE keys and values; decode at ``pos`` (= prior positions)
  writes index ``pos`` and attends over 0..pos inclusive, reading the stored BF16 values;
* logits of a stack: W_lm RMSNorm(r, gamma_final), LM head dense and BF16.
"""
from __future__ import annotations

import numpy as np

__all__ = [
    "close_mask", "index_lists", "dequantize", "bf16_bits_to_f64", "bf16_store",
    "masked_layer", "rms_norm", "rope", "softmax", "silu", "gqa_attention", "decode_layer",
    "prefill_layer", "final_logits", "decode_stack", "prefill_stack", "layer_flops",
    "active_flop_ratio", "decode_bytes",
]


# ------------------------------------------------------------------------ mask closure

def close_mask(q_keep, kv_keep, ffn_keep, group_size):
    """Dependency closure of a structured mask (Sec. "Dependency-Closed Masks and
    Cache-Consistent Routing"). Under grouped-query attention a KV group is needed exactly when at
    least one of its own query heads survives, and a head keeps its original group; a SwiGLU
    channel is a unit made of its gate row, its up row and its down column.

    Inputs are 0/1 arrays ``[L][H_q]``, ``[L][H_kv]`` (None: all kept) and ``[L][d_f]``.
    Returns boolean arrays (q', kv', ffn') with q' = q AND kv[g(h)], kv'[g] = OR_{g(h)=g} q'[h].
    """
    q = np.asarray(q_keep).astype(bool)
    L, Hq = q.shape
    Hkv = Hq // group_size
    kv_in = np.ones((L, Hkv), bool) if kv_keep is None else np.asarray(kv_keep).astype(bool)
    group_of = np.arange(Hq) // group_size
    qc = q & kv_in[:, group_of]
    kvc = np.zeros((L, Hkv), bool)
    for h in range(Hq):
        kvc[:, group_of[h]] |= qc[:, h]
    return qc, kvc, np.asarray(ffn_keep).astype(bool)


def index_lists(qc_l, kvc_l, ffnc_l, group_size):
    """Ascending retained-coordinate lists of one closed layer: query heads, KV groups, the
    KV slot (rank within the retained groups) serving each retained head, and SwiGLU channels."""
    q_idx = np.flatnonzero(qc_l).astype(np.int32)
    kv_idx = np.flatnonzero(kvc_l).astype(np.int32)
    slot_of_group = {int(g): i for i, g in enumerate(kv_idx)}
    q_kvslot = np.array([slot_of_group[int(h) // group_size] for h in q_idx], dtype=np.int32)
    ffn_idx = np.flatnonzero(ffnc_l).astype(np.int32)
    return q_idx, kv_idx, q_kvslot, ffn_idx


# ------------------------------------------------------------------------ weights

def dequantize(qw, scale):
    """W = q * s in float64 (products of an int8 and a float32 or BF16 value are exact in float64).

    ``scale`` is either one float32 value per output row, or BF16 bit patterns (uint16)
    [out][in / G] for the groupwise store: W[o][i] = q[o][i] * s[o][i // G] (paper, Table
    "configuration": symmetric groupwise INT8, group size 128, BF16 scales)."""
    q = np.asarray(qw, dtype=np.float64)
    s = np.asarray(scale)
    if s.ndim == 1:
        return q * s.astype(np.float64)[:, None]
    g = q.shape[1] // s.shape[1]
    assert g * s.shape[1] == q.shape[1]
    return q * np.repeat(bf16_bits_to_f64(s), g, axis=1)


def bf16_bits_to_f64(bits):
    b = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    return b.view(np.float32).astype(np.float64)


def bf16_store(a):
    """Value of ``a`` after storage as BF16: round to 8 significant bits, ties to even."""
    a = np.asarray(a, dtype=np.float64)
    m, e = np.frexp(a)
    return np.ldexp(np.rint(np.ldexp(m, 8)), e - 8)


def masked_layer(layer, qc_l, kvc_l, ffnc_l, head_dim):
    """Dequantised float64 weights of one layer with dropped modules zeroed.

    ``layer`` holds ``name: (int8 [out][in], float32 [out])`` for wq, wk, wv, wo, wg, wu, wd and
    BF16 bits for attn_norm / ffn_norm. Dropped query head h zeroes rows h*d_h..h*d_h+d_h-1 of
    W_q and the same columns of W_o; a dropped KV group zeroes its W_k and W_v rows; a dropped
    channel j zeroes row j of W_gate and W_up and column j of W_down.
    """
    W = {n: dequantize(*layer[n]) for n in ("wq", "wk", "wv", "wo", "wg", "wu", "wd")}
    dh = head_dim
    for h in np.flatnonzero(~np.asarray(qc_l, bool)):
        W["wq"][h * dh:(h + 1) * dh, :] = 0.0
        W["wo"][:, h * dh:(h + 1) * dh] = 0.0
    for g in np.flatnonzero(~np.asarray(kvc_l, bool)):
        W["wk"][g * dh:(g + 1) * dh, :] = 0.0
        W["wv"][g * dh:(g + 1) * dh, :] = 0.0
    drop = np.flatnonzero(~np.asarray(ffnc_l, bool))
    W["wg"][drop, :] = 0.0
    W["wu"][drop, :] = 0.0
    W["wd"][:, drop] = 0.0
    W["attn_norm"] = bf16_bits_to_f64(layer["attn_norm"])
    W["ffn_norm"] = bf16_bits_to_f64(layer["ffn_norm"])
    return W


# ------------------------------------------------------------------------ layer pieces

def rms_norm(r, gamma, eps):
    """n = r / sqrt(mean(r^2) + eps) * gamma over the last axis."""
    r = np.asarray(r, dtype=np.float64)
    return r / np.sqrt(np.mean(r * r, axis=-1, keepdims=True) + eps) * gamma


def rope(x, positions, theta):
    """Rotate-half rotary embedding of ``x [..., T, d_h]`` at integer ``positions [T]``: the
    pair (i, i + d_h/2) is rotated by the angle pos * theta^(-2i/d_h)."""
    x = np.asarray(x, dtype=np.float64)
    dh = x.shape[-1]
    half = dh // 2
    inv_freq = theta ** (-2.0 * np.arange(half, dtype=np.float64) / dh)
    ang = np.asarray(positions, dtype=np.float64)[:, None] * inv_freq[None, :]
    c, s = np.cos(ang), np.sin(ang)
    x1, x2 = x[..., :half], x[..., half:]
    return np.concatenate([x1 * c - x2 * s, x2 * c + x1 * s], axis=-1)


def softmax(s, axis=-1):
    s = np.asarray(s, dtype=np.float64)
    e = np.exp(s - np.max(s, axis=axis, keepdims=True))
    return e / np.sum(e, axis=axis, keepdims=True)


def silu(z):
    return z / (1.0 + np.exp(-z))


def gqa_attention(q, K, V, group_size, causal_offset=None):
    """Grouped-query attention. ``q [H_q][T][d_h]``, ``K, V [H_kv][n][d_h]``.

    Head h attends with its group's keys g(h) = floor(h / group_size). Scores are scaled by
    1/sqrt(d_h). With ``causal_offset`` = p0, query row t sees key positions 0..p0 + t.
    Returns ``[H_q][T][d_h]``.
    """
    Hq, T, dh = q.shape
    out = np.empty_like(q, dtype=np.float64)
    n = K.shape[1]
    for h in range(Hq):
        g = h // group_size
        s = q[h] @ K[g].T / np.sqrt(dh)                       # [T][n]
        if causal_offset is not None:
            allowed = np.arange(n)[None, :] <= (causal_offset + np.arange(T))[:, None]
            s = np.where(allowed, s, -np.inf)
        out[h] = softmax(s, axis=-1) @ V[g]
    return out


def _attention_and_ffn_inputs(W, n, sh):
    Hq, Hkv, dh = sh.n_q_heads, sh.n_kv_heads, sh.head_dim
    q = (n @ W["wq"].T).reshape(-1, Hq, dh).transpose(1, 0, 2)      # [H_q][T][d_h]
    k = (n @ W["wk"].T).reshape(-1, Hkv, dh).transpose(1, 0, 2)     # [H_kv][T][d_h]
    v = (n @ W["wv"].T).reshape(-1, Hkv, dh).transpose(1, 0, 2)
    return q, k, v


def _ffn(W, r, sh):
    n2 = rms_norm(r, W["ffn_norm"], sh.rms_eps)
    h = silu(n2 @ W["wg"].T) * (n2 @ W["wu"].T)
    return r + h @ W["wd"].T


def decode_layer(W, x, k_cache, v_cache, pos, sh, kv_store=bf16_store):
    """One decode step of one layer for a batch sharing ``pos``.

    ``x [B][d]`` residual input; ``k_cache, v_cache [B][H_kv][S][d_h]`` float64 (BF16 values),
    updated in place at index ``pos``. Returns the residual output ``[B][d]``.
    """
    x = np.asarray(x, dtype=np.float64)
    out = np.empty_like(x)
    for b in range(x.shape[0]):
        r = x[b][None, :]
        n = rms_norm(r, W["attn_norm"], sh.rms_eps)
        q, k, v = _attention_and_ffn_inputs(W, n, sh)
        q = rope(q, [pos], sh.rope_theta)
        k = rope(k, [pos], sh.rope_theta)
        k_cache[b, :, pos, :] = kv_store(k[:, 0, :])
        v_cache[b, :, pos, :] = kv_store(v[:, 0, :])
        o = gqa_attention(q, k_cache[b, :, :pos + 1], v_cache[b, :, :pos + 1], sh.group_size)
        r = r + o.transpose(1, 0, 2).reshape(1, -1) @ W["wo"].T
        out[b] = _ffn(W, r, sh)[0]
    return out


def prefill_layer(W, x, k_cache, v_cache, pos0, sh, kv_store=bf16_store):
    """Prefill of T tokens of one sequence at positions pos0..pos0+T-1, in matrix form.

    ``x [T][d]``; ``k_cache, v_cache [H_kv][S][d_h]`` updated at rows pos0..pos0+T-1. Token t
    attends causally over positions 0..pos0+t. Returns ``[T][d]``.
    """
    x = np.asarray(x, dtype=np.float64)
    T = x.shape[0]
    positions = pos0 + np.arange(T)
    n = rms_norm(x, W["attn_norm"], sh.rms_eps)
    q, k, v = _attention_and_ffn_inputs(W, n, sh)
    q = rope(q, positions, sh.rope_theta)
    k = rope(k, positions, sh.rope_theta)
    k_cache[:, pos0:pos0 + T, :] = kv_store(k)
    v_cache[:, pos0:pos0 + T, :] = kv_store(v)
    o = gqa_attention(q, k_cache[:, :pos0 + T], v_cache[:, :pos0 + T], sh.group_size,
                      causal_offset=pos0)
    r = x + o.transpose(1, 0, 2).reshape(T, -1) @ W["wo"].T
    return _ffn(W, r, sh)


def final_logits(r, final_norm_bits, lm_head_bits, eps):
    """logits = W_lm RMSNorm(r, gamma_f); W_lm is the dense BF16 LM head ``[V][d]``."""
    n = rms_norm(r, bf16_bits_to_f64(final_norm_bits), eps)
    return n @ bf16_bits_to_f64(lm_head_bits).T


def decode_stack(layer_source, closed_mask, x, caches, pos, sh, final_norm_bits=None,
                 lm_head_bits=None, kv_store=bf16_store):
    """Decode step through all layers; ``layer_source(l)`` returns layer l of the store (so
    layers can be regenerated one at a time), ``caches[l] = (K, V)``. Returns logits when an
    LM head is given, else the final residual."""
    qc, kvc, fc = closed_mask
    r = np.asarray(x, dtype=np.float64)
    for l in range(sh.n_layers):
        W = masked_layer(layer_source(l), qc[l], kvc[l], fc[l], sh.head_dim)
        r = decode_layer(W, r, caches[l][0], caches[l][1], pos, sh, kv_store)
        del W
    if lm_head_bits is None:
        return r
    return final_logits(r, final_norm_bits, lm_head_bits, sh.rms_eps)


def prefill_stack(layer_source, closed_mask, x, caches, pos0, sh, final_norm_bits=None,
                  lm_head_bits=None, kv_store=bf16_store):
    """Prefill of one sequence through all layers; ``caches[l] = (K, V)`` as ``[H_kv][S][d_h]``."""
    qc, kvc, fc = closed_mask
    r = np.asarray(x, dtype=np.float64)
    for l in range(sh.n_layers):
        W = masked_layer(layer_source(l), qc[l], kvc[l], fc[l], sh.head_dim)
        r = prefill_layer(W, r, caches[l][0], caches[l][1], pos0, sh, kv_store)
        del W
    if lm_head_bits is None:
        return r
    return final_logits(r, final_norm_bits, lm_head_bits, sh.rms_eps)


# ------------------------------------------------------------------------ ledgers

def layer_flops(sh, m_q, m_kv, c):
    """Retained per-token FLOPs of one layer, Eqs. flop-attn and flop-mlp:
    F_attn = 2 d d_h (m^q + 2 m^kv) + 2 d_h m^q d,   F_mlp = 6 d c."""
    d, dh = sh.d_model, sh.head_dim
    f_attn = 2 * d * dh * (m_q + 2 * m_kv) + 2 * dh * m_q * d
    f_mlp = 6 * d * c
    return f_attn + f_mlp


def active_flop_ratio(sh, counts):
    """Sum over layers of retained layer FLOPs over the same sum at full width; the LM head and
    embeddings are dense and left out of both sums."""
    m_q, m_kv, c = (np.asarray(a, dtype=np.int64) for a in counts)
    num = sum(layer_flops(sh, int(a), int(b), int(e)) for a, b, e in zip(m_q, m_kv, c))
    den = sh.n_layers * layer_flops(sh, sh.n_q_heads, sh.n_kv_heads, sh.d_ffn)
    return num / den


def decode_bytes(sh, counts, batch, pos, lm_head=False):
    """Algorithmic HBM bytes of one decode step: retained INT8 weights (one byte per weight,
    half the layer FLOPs), float32 scales of every computed output row (QKV rows, d O rows,
    2c gate/up rows, d down rows) and the retained BF16 KV read over pos + 1 positions. The BF16
    LM head (2 V d bytes) is added when asked."""
    d, dh = sh.d_model, sh.head_dim
    m_q, m_kv, c = (np.asarray(a, dtype=np.int64) for a in counts)
    w = sum(layer_flops(sh, int(a), int(b), int(e)) // 2 for a, b, e in zip(m_q, m_kv, c))
    s = int(sum(4 * ((a + 2 * b) * dh + d + 2 * e + d) for a, b, e in zip(m_q, m_kv, c)))
    kv = int(sum(batch * b * (pos + 1) * dh * 2 * 2 for b in m_kv))
    lm = 2 * sh.vocab * d if lm_head else 0
    return {"weights": int(w), "scales": s, "kv": kv, "lm_head": lm, "total": int(w) + s + kv + lm}


# ------------------------------------------------------------------------ request loop

def embed_rows(table, scales, ids):
    """Token embedding: row id of the INT8 table times its float32 scale (the INT8 store keeps the
    embedding dense, Sec. "Dependency-Closed Masks and Cache-Consistent Routing")."""
    ids = np.asarray(ids)
    return table[ids].astype(np.float64) * scales[ids].astype(np.float64)[:, None]


def greedy_token(logits_row):
    """Greedy decoding: the highest logit, the lowest id among equal ones."""
    return int(np.argmax(logits_row))


def generate(layer_source, closed_mask, table, scales, prompt, n_new, caches, sh,
             final_norm_bits, lm_head_bits, kv_store=bf16_store):
    """A request under one fixed plan (Sec. "Dependency-Closed Masks and Cache-Consistent
    Routing"; the timed request of Table "configuration"): prefill the prompt, take the greedy
    token of its last position, then n_new decode steps, each feeding the previous token at the
    next position. Returns the n_new + 1 generated ids and the logits they were taken from."""
    T = len(prompt)
    logits = prefill_stack(layer_source, closed_mask, embed_rows(table, scales, prompt), caches, 0,
                           sh, final_norm_bits, lm_head_bits, kv_store)
    toks, rows = [greedy_token(logits[-1])], [logits[-1]]
    for s_ in range(n_new):
        lg = decode_stack(layer_source, closed_mask, embed_rows(table, scales, [toks[-1]]),
                          [(K[None], V[None]) for K, V in caches], T + s_, sh, final_norm_bits,
                          lm_head_bits, kv_store)
        toks.append(greedy_token(lg[0]))
        rows.append(lg[0])
    return np.array(toks), np.array(rows)
