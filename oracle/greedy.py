"""Oracle for greedy dependency-closed mask construction (test infrastructure only).

Paper, Sec. "Dependency-Closed Masks and Cache-Consistent Routing": the retained set maximises the
summed predicted sensitivity under an active-FLOP budget; the implementation adds candidates
greedily by score per active FLOP and closes the GQA / SwiGLU dependencies before accepting each
addition. Candidates are query heads and SwiGLU channel groups (gate row, up row and down column
of every channel in the group, jointly). Costs follow Eqs. flop-attn and flop-mlp: a query head
costs 2 d d_h (its W_q rows) + 2 d_h d (its W_o columns); a KV group costs 2 d d_h (2 for K and
V) and is charged once, when the first of its heads is accepted; a channel group of G channels
costs 6 d G.

Readings where the paper is not explicit: the ranking key is score / active FLOPs per candidate,
where a query head carries its own cost plus 1/r of its KV group's (the group's K and V rows serve
its r heads), computed in float64 as score / (own + group / r); equal keys keep ascending
candidate index (layer-major, a layer's heads before its channel groups); in key order, a
candidate is accepted when its marginal cost (own cost, plus the whole KV group cost if the
group is not active yet) fits the remaining budget, and is skipped otherwise, in one pass. The
budget is floor(target x full-width decoder FLOPs).

Plain loops; nothing here is shared with the GPU path.
"""
from __future__ import annotations

import math

import numpy as np


def candidate_costs(sh, granule):
    """Own active-FLOP cost of a query head, of a KV group, and of a channel group."""
    d, dh = sh.d_model, sh.head_dim
    head = 2 * d * dh + 2 * dh * d
    group = 2 * d * dh * 2
    chan = 6 * d * granule
    return head, group, chan


def full_flops(sh):
    """Decoder-layer FLOPs per token at full width (sum of Eqs. flop-attn and flop-mlp)."""
    d, dh = sh.d_model, sh.head_dim
    per_layer = 2 * d * dh * (sh.n_q_heads + 2 * sh.n_kv_heads) + 2 * dh * sh.n_q_heads * d \
        + 6 * d * sh.d_ffn
    return sh.n_layers * per_layer


def budget(sh, target):
    return math.floor(target * full_flops(sh))


def candidate_list(sh, granule):
    """Candidates in index order: (layer, kind, unit) with kind 0 = query head, 1 = channel group."""
    out = []
    for l in range(sh.n_layers):
        out += [(l, 0, h) for h in range(sh.n_q_heads)]
        out += [(l, 1, g) for g in range(sh.d_ffn // granule)]
    return out


def greedy_mask(sh, head_scores, chan_scores, granule, target):
    """Returns (q_keep [L][Hq], kv_keep [L][Hkv], ffn_keep [L][F]) as uint8, the FLOPs spent and
    the accepted candidate indices in acceptance order."""
    L, Hq, Hkv, F = sh.n_layers, sh.n_q_heads, sh.n_kv_heads, sh.d_ffn
    r = Hq // Hkv
    assert F % granule == 0
    head_cost, group_cost, chan_cost = candidate_costs(sh, granule)
    cands = candidate_list(sh, granule)
    head_rank_cost = head_cost + group_cost / r            # float64, as the key
    keys = []
    for i, (l, kind, u) in enumerate(cands):
        s = float(head_scores[l][u]) if kind == 0 else float(chan_scores[l][u])
        c = head_rank_cost if kind == 0 else float(chan_cost)
        k = s / c
        keys.append((k if k != 0.0 else 0.0, i))           # one zero (no signed zeros)
    # descending key, ascending index on ties
    order = sorted(range(len(cands)), key=lambda i: (-keys[i][0], i))
    B = budget(sh, target)
    spent = 0
    q = np.zeros((L, Hq), np.uint8)
    kv = np.zeros((L, Hkv), np.uint8)
    f = np.zeros((L, F), np.uint8)
    accepted = []
    for i in order:
        l, kind, u = cands[i]
        if kind == 0:
            g = u // r
            cost = head_cost + (0 if kv[l, g] else group_cost)    # closure: the group comes along
            if spent + cost > B:
                continue
            q[l, u] = 1
            kv[l, g] = 1
        else:
            cost = chan_cost
            if spent + cost > B:
                continue
            f[l, u * granule:(u + 1) * granule] = 1
        spent += cost
        accepted.append(i)
    return q, kv, f, spent, accepted


def mask_value(sh, head_scores, chan_scores, granule, q, f):
    """Summed score of a mask (the objective)."""
    v = float((np.asarray(head_scores, np.float64) * q).sum())
    groups = f.reshape(sh.n_layers, -1, granule)[:, :, 0]
    v += float((np.asarray(chan_scores, np.float64) * groups).sum())
    return v


def mask_cost(sh, granule, q, kv, f):
    head_cost, group_cost, chan_cost = candidate_costs(sh, granule)
    return int(q.sum()) * head_cost + int(kv.sum()) * group_cost + int(f.sum()) // granule * chan_cost
