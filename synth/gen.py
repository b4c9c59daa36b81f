"""Seeded generators: INT8 per-output-channel weight store, BF16 norms / LM head / KV cache,
BF16-valued activations, and structured masks.

Every draw uses numpy's PCG64 ``default_rng`` keyed by a list, so a single layer or matrix can be
regenerated without drawing the ones before it:

* weight matrix m of layer l:  ``default_rng([seed_w, l, m])``, m = 0..6 for wq, wk, wv, wo, wg,
  wu, wd (row-major ``[out][in]``), N(0, 0.02) in float32;
* attention / FFN RMSNorm gains of layer l: ``[seed_w, l, 7]`` / ``[seed_w, l, 8]``,
  BF16(1 + 0.1 N(0, 1)), so that a missing gain multiply is visible;
* final norm gain: ``[seed_w, L, 0]``; LM head: ``[seed_w, L, 1]``, BF16(N(0, 0.02)) ``[V][d]``;
* activations: ``[seed_x]``, BF16(N(0, 1)) held in float32;
* KV cache of layer l: ``[seed_kv, l]``, BF16(N(0, 1)) for positions < pos, K drawn before V.
"""
from __future__ import annotations

import numpy as np

from .configs import Shape

__all__ = [
    "WEIGHT_NAMES", "to_bf16_bits", "bf16_bits_to_f32", "bf16_round", "quantize_rows",
    "layer_weights", "final_norm", "lm_head", "activations", "kv_prior", "tiny_mask",
    "budget_mask", "raw_mask", "all_kept_mask", "mask_counts", "embedding", "prompt_ids",
    "quantize_groups", "quantize_rows_bf16", "GROUP", "zero_dropped",
]

GROUP = 128     # columns per scale group of the groupwise store

WEIGHT_NAMES = ("wq", "wk", "wv", "wo", "wg", "wu", "wd")


def to_bf16_bits(a) -> np.ndarray:
    """float32 -> BF16 bit patterns (uint16), round to nearest even; NaN stays NaN."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    u = a.view(np.uint32)
    lsb = (u >> np.uint32(16)) & np.uint32(1)
    r = ((u + np.uint32(0x7FFF) + lsb) >> np.uint32(16)).astype(np.uint16)
    nan = np.isnan(a)
    if nan.any():
        r[nan] = np.uint16(0x7FC0)
    return r


def bf16_bits_to_f32(b) -> np.ndarray:
    b = np.ascontiguousarray(b, dtype=np.uint16)
    return (b.astype(np.uint32) << np.uint32(16)).view(np.float32)


def bf16_round(a) -> np.ndarray:
    """float32 values rounded to the nearest BF16 value, returned as float32."""
    return bf16_bits_to_f32(to_bf16_bits(a))


def quantize_rows(w: np.ndarray):
    """Symmetric per-output-row INT8: s_r = max_k |w_rk| / 127 (float32, 1 for an all-zero
    row), q = clip(rint(w / s_r), -127, 127) with ties to even."""
    w = np.asarray(w, dtype=np.float32)
    amax = np.abs(w).max(axis=1)
    s = (amax / np.float32(127.0)).astype(np.float32)
    s[amax == 0] = np.float32(1.0)
    q = np.rint(w / s[:, None])
    np.clip(q, -127, 127, out=q)
    return q.astype(np.int8), s


def quantize_rows_bf16(w: np.ndarray):
    """Per-output-row INT8 whose scales are BF16 values: s_r = BF16(max_k |w_rk| / 127) (1 for an
    all-zero row), q = clip(rint(w / s_r), -127, 127). Returns (int8 [out][in], float32 [out]);
    the same bytes with every group scale equal to s_r form a groupwise store of identical
    quantisation."""
    w = np.asarray(w, dtype=np.float32)
    amax = np.abs(w).max(axis=1)
    s = bf16_round((amax / np.float32(127.0)).astype(np.float32))
    s[amax == 0] = np.float32(1.0)
    q = np.rint(w / s[:, None])
    np.clip(q, -127, 127, out=q)
    return q.astype(np.int8), s


def quantize_groups(w: np.ndarray, group: int = GROUP):
    """Symmetric groupwise INT8 with BF16 scales: for row r and each run g of ``group``
    consecutive columns, s = BF16(max |w| / 127) (1 for an all-zero run) and q = clip(rint(w / s),
    -127, 127), ties to even (a scale rounded below max/127 clips the largest entries at 127).
    Returns (int8 [out][in], uint16 BF16 bits [out][in / group])."""
    w = np.asarray(w, dtype=np.float32)
    o, i = w.shape
    assert i % group == 0, (i, group)
    wg = w.reshape(o, i // group, group)
    amax = np.abs(wg).max(axis=2)
    s = bf16_round((amax / np.float32(127.0)).astype(np.float32))
    s[amax == 0] = np.float32(1.0)
    q = np.rint(wg / s[:, :, None])
    np.clip(q, -127, 127, out=q)
    return q.reshape(o, i).astype(np.int8), to_bf16_bits(s)


def _weight_shapes(sh: Shape):
    qd, kd = sh.n_q_heads * sh.head_dim, sh.n_kv_heads * sh.head_dim
    d, f = sh.d_model, sh.d_ffn
    return {"wq": (qd, d), "wk": (kd, d), "wv": (kd, d), "wo": (d, qd),
            "wg": (f, d), "wu": (f, d), "wd": (d, f)}


def _gain(rng, n):
    return to_bf16_bits(np.float32(1.0) + np.float32(0.1) * rng.standard_normal(n, dtype=np.float32))


def layer_weights(sh: Shape, layer: int, seed_w: int = 0, std: float = 0.02,
                  quant: str = "row") -> dict:
    """One decoder layer of the INT8 store.

    Returns ``{name: (int8 [out][in], scales)}`` for the seven projections plus ``attn_norm`` /
    ``ffn_norm`` as BF16 bit patterns ``uint16 [d]``. ``quant``: "row" (float32 scale per row),
    "row_bf16" (per row, BF16-valued float32 scales) or "group" (BF16 bits [out][in / 128]). The
    float weights drawn are the same for every ``quant``.
    """
    qz = {"row": quantize_rows, "row_bf16": quantize_rows_bf16, "group": quantize_groups}[quant]
    out = {}
    for m, (name, shp) in enumerate(_weight_shapes(sh).items()):
        rng = np.random.default_rng([seed_w, layer, m])
        w = rng.standard_normal(shp, dtype=np.float32)
        w *= np.float32(std)
        out[name] = qz(w)
        del w
    out["attn_norm"] = _gain(np.random.default_rng([seed_w, layer, 7]), sh.d_model)
    out["ffn_norm"] = _gain(np.random.default_rng([seed_w, layer, 8]), sh.d_model)
    return out


def final_norm(sh: Shape, seed_w: int = 0) -> np.ndarray:
    return _gain(np.random.default_rng([seed_w, sh.n_layers, 0]), sh.d_model)


def lm_head(sh: Shape, seed_w: int = 0, std: float = 0.02) -> np.ndarray:
    """BF16 bit patterns ``uint16 [V][d]``."""
    rng = np.random.default_rng([seed_w, sh.n_layers, 1])
    w = rng.standard_normal((sh.vocab, sh.d_model), dtype=np.float32)
    w *= np.float32(std)
    return to_bf16_bits(w)


def embedding(sh: Shape, seed_w: int = 0):
    """INT8 token embedding ``(int8 [V][d], float32 [V])``: N(0, 1) rows quantised per row."""
    rng = np.random.default_rng([seed_w, sh.n_layers, 2])
    w = rng.standard_normal((sh.vocab, sh.d_model), dtype=np.float32)
    return quantize_rows(w)


def prompt_ids(n: int, vocab: int, seed: int = 4) -> np.ndarray:
    """Seeded prompt token ids, int32 [n], uniform over the vocabulary."""
    return np.random.default_rng([seed]).integers(0, vocab, n).astype(np.int32)


def activations(n_rows: int, d: int, seed_x: int = 1) -> np.ndarray:
    """BF16-valued N(0, 1) rows ``float32 [n_rows][d]``."""
    rng = np.random.default_rng([seed_x])
    return bf16_round(rng.standard_normal((n_rows, d), dtype=np.float32))


def kv_prior(sh: Shape, layer: int, batch: int, pos: int, max_seq: int, seed_kv: int = 2,
             fill: float = 0.0):
    """Prior K and V cache contents of one layer as BF16 bits ``uint16 [B][Hkv][S][dh]``.

    Positions < pos hold BF16(N(0, 1)) draws (treated as already rotated keys); positions
    >= pos hold ``fill`` (use NaN to prove that unwritten rows are never read).
    """
    rng = np.random.default_rng([seed_kv, layer])
    shp = (batch, sh.n_kv_heads, pos, sh.head_dim)
    kd = rng.standard_normal(shp, dtype=np.float32)
    vd = rng.standard_normal(shp, dtype=np.float32)
    full = (batch, sh.n_kv_heads, max_seq, sh.head_dim)
    fill_bits = to_bf16_bits(np.array([fill], dtype=np.float32))[0]
    k = np.full(full, fill_bits, dtype=np.uint16)
    v = np.full(full, fill_bits, dtype=np.uint16)
    k[:, :, :pos] = to_bf16_bits(kd)
    v[:, :, :pos] = to_bf16_bits(vd)
    return k, v


# ----------------------------------------------------------------------------------- masks

def all_kept_mask(sh: Shape):
    L = sh.n_layers
    return (np.ones((L, sh.n_q_heads), np.uint8), np.ones((L, sh.n_kv_heads), np.uint8),
            np.ones((L, sh.d_ffn), np.uint8))


def tiny_mask(sh: Shape, seed: int = 1):
    """Drops 2 of 8 query heads (both KV groups stay) and keeps 1024 of 1536 FFN channels,
    per layer, from ``default_rng(seed)``."""
    rng = np.random.default_rng(seed)
    q, kv, f = all_kept_mask(sh)
    f[:] = 0
    for l in range(sh.n_layers):
        drop = rng.choice(sh.n_q_heads, 2, replace=False)
        q[l, drop] = 0
        keep = np.sort(rng.choice(sh.d_ffn, sh.d_ffn * 2 // 3, replace=False))
        f[l, keep] = 1
    return q, kv, f


def raw_mask(sh: Shape, seed: int, p_q=0.7, p_kv=0.8, p_f=0.6, block: int = 1):
    """Independent Bernoulli keep bits per query head, KV group and FFN channel. The result is
    generally not dependency-closed (a kept head may sit in a dropped group, a kept group may
    have no kept head), which exercises the closure. With ``block`` > 1 the FFN bits are drawn
    per aligned block of that many channels."""
    rng = np.random.default_rng([seed, 77])
    L = sh.n_layers
    q = (rng.uniform(size=(L, sh.n_q_heads)) < p_q).astype(np.uint8)
    kv = (rng.uniform(size=(L, sh.n_kv_heads)) < p_kv).astype(np.uint8)
    if block > 1:
        fb = (rng.uniform(size=(L, sh.d_ffn // block)) < p_f).astype(np.uint8)
        return q, kv, np.repeat(fb, block, axis=1)
    f = (rng.uniform(size=(L, sh.d_ffn)) < p_f).astype(np.uint8)
    return q, kv, f


def zero_dropped(layer: dict, sh: Shape, q_keep, kv_keep, f_keep) -> dict:
    """A copy of one layer of the INT8 store in which the weights of dropped modules are zero and
    every scale is unchanged: the W_q rows of each dropped query head and the W_o columns that
    read it, the W_k and W_v rows of each dropped KV group, and the gate row, up row and W_down
    column of each dropped FFN channel. ``*_keep`` are one layer's dependency-closed keep bits.
    Dequantised, this is the zero-masked layer, so a dense plan over it computes the masked layer
    with the dense launch shapes (the mask-as-zero control)."""
    dh = sh.head_dim
    dq = np.repeat(~np.asarray(q_keep, bool), dh)
    dkv = np.repeat(~np.asarray(kv_keep, bool), dh)
    df = ~np.asarray(f_keep, bool)
    out = dict(layer)
    for name, rows, cols in (("wq", dq, None), ("wk", dkv, None), ("wv", dkv, None),
                             ("wo", None, dq), ("wg", df, None), ("wu", df, None),
                             ("wd", None, df)):
        w, sc = layer[name]
        w = w.copy()
        if rows is not None:
            w[rows, :] = 0
        if cols is not None:
            w[:, cols] = 0
        out[name] = (w, sc)
    return out


def mask_counts(q, kv, f):
    """Kept query heads, KV groups and FFN channels per layer of a closed mask."""
    return q.sum(axis=1), kv.sum(axis=1), f.sum(axis=1)


def budget_mask(sh: Shape, seed: int, target: float = 0.57, granule: int = 128):
    """A structured mask at an active-FLOP budget, drawn per candidate.

    Stands in for the offline mask construction, which is not part of the decode path. Keep
    probabilities are drawn uniformly in [0.3, 1] per KV group, per query head and per FFN
    granule of ``granule`` channels, then scaled by one factor (bisection) so that the
    expected active FLOPs equal ``target`` x dense. Groups, heads and granules are then kept by
    uniform draws; a head needs its group, and a group with no kept head is dropped. Finally
    FFN granules are dropped in ascending keep probability while over budget, and added back in
    descending order while one still fits. The result is dependency-closed by construction.
    """
    L, Hq, Hkv = sh.n_layers, sh.n_q_heads, sh.n_kv_heads
    d, dh, F, r = sh.d_model, sh.head_dim, sh.d_ffn, sh.group_size
    G = granule
    assert F % G == 0
    nG = F // G
    rng = np.random.default_rng(seed)
    p_grp = rng.uniform(0.3, 1.0, (L, Hkv))
    p_head = rng.uniform(0.3, 1.0, (L, Hq))
    p_ffn = rng.uniform(0.3, 1.0, (L, nG))
    unit = 4 * d * dh            # one query head or one KV group: its projection rows + columns
    granule_cost = 6 * d * G      # one FFN granule: gate row, up row and down column per channel
    dense = L * (unit * (Hq + Hkv) + 6 * d * F)
    budget = target * dense

    def expected(s):
        kg = np.minimum(1.0, s * p_grp)
        kh = np.minimum(1.0, s * p_head).reshape(L, Hkv, r)
        kf = np.minimum(1.0, s * p_ffn)
        return unit * float((kg * (1.0 + kh.sum(axis=2))).sum()) + granule_cost * float(kf.sum())

    lo, hi = 0.0, 1.0 / 0.3
    for _ in range(80):
        mid = 0.5 * (lo + hi)
        if expected(mid) > budget:
            hi = mid
        else:
            lo = mid
    s = lo
    kg = np.minimum(1.0, s * p_grp)
    kh = np.minimum(1.0, s * p_head)
    kf = np.minimum(1.0, s * p_ffn)
    u_grp = rng.uniform(size=(L, Hkv))
    u_head = rng.uniform(size=(L, Hq))
    u_ffn = rng.uniform(size=(L, nG))
    grp = u_grp < kg
    head = (u_head < kh) & np.repeat(grp, r, axis=1)
    grp = grp & head.reshape(L, Hkv, r).any(axis=2)
    ffn_g = u_ffn < kf

    attn_cost = unit * (int(head.sum()) + int(grp.sum()))
    cost = attn_cost + granule_cost * int(ffn_g.sum())
    flat = np.arange(L * nG)
    pf = p_ffn.ravel()
    fg = ffn_g.ravel()
    for idx in np.lexsort((flat, pf)):          # ascending probability, ties by index
        if cost <= budget:
            break
        if fg[idx]:
            fg[idx] = False
            cost -= granule_cost
    for idx in np.lexsort((flat, -pf)):         # descending probability, ties by index
        if not fg[idx] and cost + granule_cost <= budget:
            fg[idx] = True
            cost += granule_cost
    ffn = np.repeat(fg.reshape(L, nG), G, axis=1)
    return head.astype(np.uint8), grp.astype(np.uint8), ffn.astype(np.uint8)
