"""Fourth CPU reference: pure-Python scalar loops for very small layers.

TEST INFRASTRUCTURE ONLY (see ``oracle.reference``). The mask is applied by structural removal
(loops run over retained heads and channels only), not by zeroing, and every sum is an explicit
loop over Python floats, so it shares neither mechanism nor library calls with the oracle.
"""
from __future__ import annotations

import math

__all__ = ["scalar_decode_layer"]


def _bf16(v):
    if v == 0.0:
        return 0.0
    m, e = math.frexp(v)
    return math.ldexp(round(m * 256.0), e - 8)     # round() is ties-to-even


def scalar_decode_layer(layer, keep_q, keep_kv, keep_f, x, kc, vc, pos, sh, round_cache=True):
    """``layer``: name -> (int8 rows as lists, scale list), gains as Python floats lists.
    ``keep_*``: closed masks of this layer as lists of bools. ``x``: list of floats.
    ``kc, vc``: nested lists [H_kv][S][d_h] updated in place. Returns the output list."""
    d, dh, Hq = sh.d_model, sh.head_dim, sh.n_q_heads
    r = sh.n_q_heads // sh.n_kv_heads

    def mat_row(name, row, vec):
        qrow, s = layer[name][0][row], layer[name][1][row]
        acc = 0.0
        for j in range(len(vec)):
            acc += float(qrow[j]) * float(s) * vec[j]
        return acc

    def norm(vec, g):
        ms = 0.0
        for v in vec:
            ms += v * v
        inv = 1.0 / math.sqrt(ms / len(vec) + sh.rms_eps)
        return [vec[i] * inv * g[i] for i in range(len(vec))]

    def rot(vec):
        half = dh // 2
        outv = [0.0] * dh
        for i in range(half):
            ang = pos * sh.rope_theta ** (-2.0 * i / dh)
            c, s = math.cos(ang), math.sin(ang)
            outv[i] = vec[i] * c - vec[i + half] * s
            outv[i + half] = vec[i + half] * c + vec[i] * s
        return outv

    n = norm(x, layer["attn_norm"])
    for g in range(sh.n_kv_heads):
        if not keep_kv[g]:
            continue
        k = rot([mat_row("wk", g * dh + e, n) for e in range(dh)])
        v = [mat_row("wv", g * dh + e, n) for e in range(dh)]
        for e in range(dh):
            kc[g][pos][e] = _bf16(k[e]) if round_cache else k[e]
            vc[g][pos][e] = _bf16(v[e]) if round_cache else v[e]
    attn = [0.0] * (Hq * dh)
    for h in range(Hq):
        if not keep_q[h]:
            continue
        g = h // r
        q = rot([mat_row("wq", h * dh + e, n) for e in range(dh)])
        scores = []
        for t in range(pos + 1):
            acc = 0.0
            for e in range(dh):
                acc += q[e] * kc[g][t][e]
            scores.append(acc / math.sqrt(dh))
        mx = max(scores)
        w = [math.exp(s - mx) for s in scores]
        tot = sum(w)
        for e in range(dh):
            acc = 0.0
            for t in range(pos + 1):
                acc += w[t] / tot * vc[g][t][e]
            attn[h * dh + e] = acc
    h1 = [x[i] + mat_row("wo", i, attn) for i in range(d)]
    f = norm(h1, layer["ffn_norm"])
    hidden = {}
    for j in range(sh.d_ffn):
        if not keep_f[j]:
            continue
        gt = mat_row("wg", j, f)
        hidden[j] = gt / (1.0 + math.exp(-gt)) * mat_row("wu", j, f)
    out = []
    for i in range(d):
        qrow, s = layer["wd"][0][i], layer["wd"][1][i]
        acc = 0.0
        for j, hv in hidden.items():
            acc += float(qrow[j]) * float(s) * hv
        out.append(h1[i] + acc)
    return out
